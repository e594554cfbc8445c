"""C ABI checks that need no GPU: the library loads and exports every entry
point its header declares; the host tree builder is bit-exact against the
oracle; host-side validation rejects bad arguments before any device work."""
import ctypes as C
import os
import re

import numpy as np
import pytest

import oracle as O
import paper_2405_18628_amd as ppd
from synth.trees import make_tree

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    hdr = open(os.path.join(ROOT, "include", "ppd.h")).read()
    return sorted(set(re.findall(r"\b(ppd_[a-z_]+)\s*\(", hdr)))


def test_library_exports_every_declared_symbol():
    L = ppd.lib()
    names = _declared()
    assert {"ppd_verify_step", "ppd_accept", "ppd_kv_compact", "ppd_build_tree_mask"} <= set(names)
    for n in names:
        assert hasattr(L, n), n


@pytest.mark.parametrize("spec", ["candidates:10", "candidates:32", "total:64", "total:128",
                                  "chain:128", "chain:1"])
def test_build_tree_mask_bit_exact(spec):
    for seed in range(20):
        if spec.startswith("chain"):
            n = int(spec.split(":")[1])
            parent = [-1] + list(range(n - 1))
        else:
            parent = make_tree(spec, 1000, 3, 5, seed, 1).parent
        depth, mask = ppd.ppd_build_tree_mask(parent)
        od, anc = O.build_mask(parent)
        assert np.array_equal(depth, od.astype(np.int32))
        assert np.array_equal(mask, O.pack_mask(anc))
        if spec.startswith("chain"):
            break


@pytest.mark.parametrize("parent,code", [([0], ppd.PPD_ETREE), ([-1, 1], ppd.PPD_ETREE),
                                         ([-1, 0, 3], ppd.PPD_ETREE), ([-1, -1], ppd.PPD_ETREE),
                                         ([], ppd.PPD_EINVAL),
                                         ([-1] + list(range(128)), ppd.PPD_EINVAL)])
def test_build_tree_mask_rejects(parent, code):
    with pytest.raises(ppd.PPDError) as e:
        ppd.ppd_build_tree_mask(parent)
    assert e.value.status == code


def _fake_model(dtype=ppd.PPD_BF16, **kw):
    """A model description whose pointers are non-null but never dereferenced:
    every call below fails validation (or is host-only) before device work."""
    n = kw.get("n_layers", 2)
    fake = C.c_void_p(0x1000)
    arr = (C.c_void_p * n)(*([0x1000] * n))
    keep = [arr]
    m = ppd.ppd_model(n, kw.get("hidden", 512), kw.get("n_heads", 4), kw.get("n_kv_heads", 4),
                      kw.get("head_dim", 128), kw.get("ffn", 1344), kw.get("vocab", 1000), 3,
                      1e-6, 10000.0, dtype, fake, fake,
                      *[C.cast(arr, C.POINTER(C.c_void_p)) for _ in range(6)], fake, fake)
    return m, keep


def test_workspace_bytes_and_model_validation():
    L = ppd.lib()
    m, keep = _fake_model()
    n64 = L.ppd_workspace_bytes(C.byref(m), 64, 4096)
    n128 = L.ppd_workspace_bytes(C.byref(m), 128, 4096)
    assert 0 < n64 <= n128
    assert L.ppd_workspace_bytes(C.byref(m), 0, 10) == 0
    assert L.ppd_workspace_bytes(C.byref(m), 129, 10) == 0
    for bad in (dict(head_dim=64), dict(hidden=500), dict(ffn=1000), dict(n_kv_heads=3)):
        mb, kb = _fake_model(**bad)
        assert L.ppd_workspace_bytes(C.byref(mb), 16, 10) == 0
        assert ppd.ppd_last_error()
    mf, kf = _fake_model(ppd.PPD_F32, head_dim=64, hidden=256, ffn=688)
    assert L.ppd_workspace_bytes(C.byref(mf), 40, 200) > 0


def test_verify_rejects_before_enqueue():
    L = ppd.lib()
    m, keep = _fake_model()
    kv = ppd.ppd_kv(0x2000, 0x3000, 256, None)
    fake = 0x4000
    ws_bytes = L.ppd_workspace_bytes(C.byref(m), 16, 256)

    def call(T=16, Lc=0, kvd=kv, wsb=ws_bytes, ids=fake):
        return L.ppd_verify_step(C.byref(m), C.byref(kvd), Lc, T, ids, fake, fake, fake, wsb,
                                 None, fake, None)
    assert call(T=0) == ppd.PPD_EINVAL
    assert call(T=129) == ppd.PPD_EINVAL
    assert call(Lc=-1) == ppd.PPD_EINVAL
    assert call(Lc=250) == ppd.PPD_ECAPACITY
    assert call(wsb=ws_bytes - 1) == ppd.PPD_EWORKSPACE
    assert call(ids=None) == ppd.PPD_EINVAL
    assert call(kvd=ppd.ppd_kv(0x2000, 0x3000, 252, None)) == ppd.PPD_EUNSUPPORTED
    assert call(kvd=ppd.ppd_kv(None, 0x3000, 256, None)) == ppd.PPD_EINVAL
    assert "capacity" in ppd.ppd_last_error() or ppd.ppd_last_error()


def test_accept_and_compact_reject_before_enqueue():
    L = ppd.lib()
    m, keep = _fake_model()
    f = 0x4000
    assert L.ppd_accept(0, f, f, f, 10, f, f, f, f, 64, None) == ppd.PPD_EINVAL
    assert L.ppd_accept(129, f, f, f, 10, f, f, f, f, 64, None) == ppd.PPD_EINVAL
    assert L.ppd_accept(4, f, f, f, 0, f, f, f, f, 64, None) == ppd.PPD_EINVAL
    assert L.ppd_accept(4, f, f, f, 10, f, f, f, None, 64, None) == ppd.PPD_EWORKSPACE
    kv = ppd.ppd_kv(0x2000, 0x3000, 256, None)
    assert L.ppd_kv_compact(C.byref(m), C.byref(kv), 256, f, 4, f, None) == ppd.PPD_ECAPACITY
    assert L.ppd_kv_compact(C.byref(m), C.byref(kv), 10, None, 4, f, None) == ppd.PPD_EINVAL
    assert L.ppd_kv_compact(C.byref(m), C.byref(kv), 10, f, 0, f, None) == ppd.PPD_EINVAL
    assert L.ppd_kv_compact(C.byref(m), C.byref(kv), 10, f, 129, f, None) == ppd.PPD_EINVAL
    assert L.ppd_workspace_init(None, 0, None) == ppd.PPD_EWORKSPACE


def test_packed_weight_sizes_and_rejections():
    """Packed size = groups of 16 output rows (gate/up: 16 features, i.e. 32
    rows) x columns x 2 bytes: the matrix itself, plus zero rows up to a
    whole group (the LM head's vocabulary, a ragged feature count)."""
    L = ppd.lib()
    cases = [(ppd.PPD_W_QKV, 3 * 4096, 4096, 3 * 4096), (ppd.PPD_W_O, 4096, 4096, 4096),
             (ppd.PPD_W_GATE_UP, 2 * 11008, 4096, 2 * 11008), (ppd.PPD_W_GATE_UP, 2 * 13824, 5120, 2 * 13824),
             (ppd.PPD_W_QKV, 3 * 5120, 5120, 3 * 5120), (ppd.PPD_W_DOWN, 4096, 11008, 4096),
             (ppd.PPD_W_LM_HEAD, 32000, 4096, 32000), (ppd.PPD_W_LM_HEAD, 1000, 512, 1008),
             (ppd.PPD_W_LM_HEAD, 37, 64, 48), (ppd.PPD_W_DOWN, 512, 1344, 512),
             (ppd.PPD_W_GATE_UP, 2 * 1344, 512, 2 * 1344)]
    for kind, rows, cols, padded_rows in cases:
        assert ppd.ppd_packed_weight_bytes(kind, rows, cols) == padded_rows * cols * 2, (kind, rows, cols)
    for kind, rows, cols in [(ppd.PPD_W_QKV, 3 * 4096, 4000), (ppd.PPD_W_QKV, 3 * 4096 - 64, 4096),
                             (ppd.PPD_W_O, 4000, 4096), (ppd.PPD_W_GATE_UP, 2 * 1000, 512),
                             (ppd.PPD_W_LM_HEAD, 0, 512), (5, 128, 128), (-1, 128, 128)]:
        assert L.ppd_packed_weight_bytes(kind, rows, cols) == 0
        assert ppd.ppd_last_error()
    f = 0x4000
    assert L.ppd_pack_weight(ppd.PPD_W_O, 512, 512, None, f, None) == ppd.PPD_EINVAL
    assert L.ppd_pack_weight(ppd.PPD_W_O, 512, 512, f, None, None) == ppd.PPD_EINVAL
    assert L.ppd_pack_weight(ppd.PPD_W_O, 500, 512, f, f, None) == ppd.PPD_EUNSUPPORTED
    assert L.ppd_pack_weight(9, 512, 512, f, f, None) == ppd.PPD_EINVAL
    # a packed weight is read through one buffer resource: at most 0x7ffffff0
    # bytes (2^30 - 8 rows of 1024 bf16 columns fit, 2^30 do not)
    ok_rows = (0x7ffffff0 // (2 * 1024)) // 16 * 16
    assert ppd.ppd_packed_weight_bytes(ppd.PPD_W_LM_HEAD, ok_rows, 1024) == ok_rows * 1024 * 2
    assert L.ppd_packed_weight_bytes(ppd.PPD_W_LM_HEAD, 1 << 20, 1024) == 0
    assert L.ppd_pack_weight(ppd.PPD_W_LM_HEAD, 1 << 20, 1024, f, f, None) == ppd.PPD_EUNSUPPORTED


def test_next_tree_rejects_before_enqueue():
    """Template and argument checks of ppd_next_tree (host side, nothing is
    enqueued on failure)."""
    import numpy as np
    L = ppd.lib()
    f = 0x4000

    def call(tp, tk, T=8, vocab=100, n_prompt=3, ws=f, wsb=64, logits=f, n_ept=1):
        tp = np.asarray(tp, np.int32)
        tk = np.asarray(tk, np.int32)
        return L.ppd_next_tree(T, f, f, vocab, n_prompt, n_ept, logits, f, f, f, len(tp),
                               tp.ctypes.data, tk.ctypes.data, f, ws, wsb, None)
    assert call([0, 0], [0, 0]) == ppd.PPD_EINVAL                  # root not -1
    assert call([-1, 1], [0, 0]) == ppd.PPD_EINVAL                 # not topological
    assert call([-1, 0, 1], [0, -1, 0]) == ppd.PPD_EINVAL          # candidate under prompt
    assert call([-1, 0, 0], [0, 0, -2]) == ppd.PPD_EINVAL          # prompt 1 under root
    assert call([-1, 0], [0, 16]) == ppd.PPD_EINVAL                # rank >= PPD_TOPK_MAX
    assert call([-1, 0], [0, 5], vocab=5) == ppd.PPD_EINVAL        # rank >= vocab
    assert call([-1, 0], [0, -4]) == ppd.PPD_EINVAL                # prompt id >= n_prompt
    deep = [-1] + list(range(16))
    assert call(deep, [0] * 17) == ppd.PPD_EINVAL                  # depth 16 > 15
    assert call([-1, 0], [0, 0], T=0) == ppd.PPD_EINVAL
    assert call([-1, 0], [0, 0], T=129) == ppd.PPD_EINVAL
    assert call([-1, 0], [0, 0], ws=None) == ppd.PPD_EWORKSPACE
    assert call([-1, 0], [0, 0], logits=None) == ppd.PPD_EINVAL
    assert call(list(range(-1, 128)), [0] * 129) == ppd.PPD_EINVAL  # template > PPD_T_MAX
    assert "template" in ppd.ppd_last_error()
    # ensemble prompt tokens: group g's chain continues with group g only
    assert call([-1, 0], [0, 0], n_ept=0) == ppd.PPD_EINVAL
    assert call([-1, 0], [0, 0], n_ept=65) == ppd.PPD_EINVAL       # > PPD_EPT_MAX
    assert call([-1, 0, 1], [0, -1, -4], n_ept=2) == ppd.PPD_EINVAL  # group 0 then group 1
    assert call([-1, 0, 1], [0, -2, -3], n_ept=2) == ppd.PPD_EINVAL  # group 1 then group 0
    assert call([-1, 0], [0, -7], n_ept=2) == ppd.PPD_EINVAL         # token distance 4 > 3
    assert call([-1, 0, 0], [0, 0, -3], n_ept=2) == ppd.PPD_EINVAL   # distance 2 under the root


@pytest.mark.parametrize("depth_max,k_max,n_cand,n_prompt,n_ept,seed", [
    (3, 16, 15, 3, 1, 0), (3, 16, 31, 3, 1, 1), (3, 16, 0, 3, 1, 2), (2, 3, 12, 2, 1, 3),
    (4, 5, 20, 3, 1, 4), (3, 16, 7, 3, 2, 5), (1, 16, 16, 3, 1, 6), (3, 16, 24, 3, 1, 7),
])
def test_sparse_template_matches_oracle(depth_max, k_max, n_cand, n_prompt, n_ept, seed):
    """The host tree-sizing builder against the oracle's listing of every
    rank path: the same template, bit-exact, and the same Proposition-1
    value.  Tables: the synthetic one, random ones, and rows with ties."""
    from synth.trees import synthetic_accept_table
    rng = np.random.default_rng(seed)
    if seed == 0 or seed == 1 or seed == 2:
        p = synthetic_accept_table(depth_max, k_max)
    elif seed == 7:
        p = np.round(rng.random((depth_max, k_max)) * 4) / 4   # many equal products
    else:
        p = rng.random((depth_max, k_max))
    tp, tk, f = ppd.ppd_sparse_template(p, n_cand, n_prompt, n_ept)
    rp, rk, rf = O.sparse_template(p, n_cand, n_prompt, n_ept)
    assert tp.tolist() == rp.tolist() and tk.tolist() == rk.tolist()
    assert f == rf


def test_sparse_template_rejects():
    p = np.full((3, 16), 0.1)
    for bad in (dict(p_table=np.full((3, 16), 1.5)), dict(p_table=np.full((3, 16), np.nan)),
                dict(p_table=np.full((16, 4), 0.1)), dict(p_table=np.full((3, 17), 0.1)),
                dict(n_cand=32), dict(n_cand=-1), dict(n_ept=0),
                dict(p_table=np.full((1, 2), 0.5), n_cand=3, n_prompt=1)):
        args = dict(p_table=p, n_cand=10, n_prompt=3, n_ept=1)
        args.update(bad)
        with pytest.raises(ppd.PPDError):
            ppd.ppd_sparse_template(args["p_table"], args["n_cand"], args["n_prompt"],
                                    args["n_ept"])


def test_verify_batch_rejects_before_enqueue():
    L = ppd.lib()
    m, keep = _fake_model()
    fake = 0x4000
    ws_bytes = L.ppd_workspace_bytes(C.byref(m), 128, 256)

    def call(Ls, Ts, caps=None, B=None, wsb=ws_bytes, model=m):
        B = len(Ls) if B is None else B
        n = max(1, len(Ls))
        kvs = (ppd.ppd_kv * n)(*[ppd.ppd_kv(0x2000, 0x3000, (caps or [256] * n)[j], None)
                                 for j in range(n)])
        La = np.asarray(Ls + [0] * (n - len(Ls)), np.int32)
        Ta = np.asarray(Ts + [0] * (n - len(Ts)), np.int32)
        return L.ppd_verify_batch(C.byref(model), B, C.cast(kvs, C.c_void_p), La.ctypes.data,
                                  Ta.ctypes.data, fake, fake, fake, fake, wsb, None, fake, None)
    assert call([0, 0], [16, 16], B=0) == ppd.PPD_EINVAL
    assert call([0] * 17, [4] * 17) == ppd.PPD_EINVAL                 # B > PPD_BATCH_MAX
    assert call([0, 0, 0], [64, 64, 1]) == ppd.PPD_EINVAL             # 129 tokens in all
    assert call([0, 0], [16, 0]) == ppd.PPD_EINVAL                    # an empty tree
    assert call([0, -1], [16, 16]) == ppd.PPD_EINVAL
    assert call([0, 250], [16, 16]) == ppd.PPD_ECAPACITY             # sequence 1 overflows
    assert call([0, 0], [16, 16], caps=[256, 252]) == ppd.PPD_EUNSUPPORTED
    assert call([0, 0], [64, 64], wsb=ws_bytes - 1) == ppd.PPD_EWORKSPACE
    mf, kf = _fake_model(ppd.PPD_F32, head_dim=64, hidden=256, ffn=688)
    assert call([0, 0], [8, 8], model=mf) == ppd.PPD_EUNSUPPORTED       # batches need bf16


def test_read_probe_rejects_before_enqueue():
    """The HBM read probe checks its arguments on the host."""
    L = ppd.lib()
    f = 0x4000
    assert L.ppd_read_probe(None, 16, f, None) == ppd.PPD_EINVAL
    assert L.ppd_read_probe(f, 16, None, None) == ppd.PPD_EINVAL
    assert L.ppd_read_probe(f, 24, f, None) == ppd.PPD_EINVAL
    assert L.ppd_read_probe(f + 4, 16, f, None) == ppd.PPD_EINVAL
