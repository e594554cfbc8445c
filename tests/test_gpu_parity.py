"""GPU parity: the HIP verification step, acceptance and compaction against
the CPU oracle on the same seeded inputs (see gpu_cases for the rules)."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2405_18628_amd as ppd
from gpu_cases import (check_logits, check_pred, gpu_step, make_case, oracle_step, say,
                       subtree, tree_for, workspace)
from synth import workload
from synth.trees import Tree, make_tree

pytestmark = pytest.mark.gpu


def _accept_and_compact(case, tree, res, ws):
    """GPU accept on the GPU's greedy tokens == oracle accept on them; the
    compaction moves exactly the accepted rows (bit-exact)."""
    T = tree.T
    tt = res["tt"]
    pred_dev = torch.from_numpy(res["pred"].astype(np.int32)).cuda()
    path = torch.full((T,), -7, dtype=torch.int32, device="cuda")
    n_path = torch.zeros(1, dtype=torch.int32, device="cuda")
    nxt = torch.zeros(1, dtype=torch.int32, device="cuda")
    ppd.ppd_accept(T, tt["parent"], tt["ids"], pred_dev, case.shape.vocab, path, n_path, nxt, ws)
    torch.cuda.synchronize()
    opath, on, onext = O.accept(tree.parent, tree.ids, res["pred"], case.shape.vocab)
    n = int(n_path.item())
    assert n == on and int(nxt.item()) == onext
    assert path[:n].cpu().tolist() == list(opath)
    L = case.L
    k_before = case.k.clone()
    v_before = case.v.clone()
    len_dev = torch.zeros(1, dtype=torch.int32, device="cuda")
    ppd.ppd_kv_compact(case.model, ppd.KVCache(case.k, case.v, len_dev), L, path, n_path)
    torch.cuda.synchronize()
    assert int(len_dev.item()) == L + n
    idx = torch.tensor(list(opath), device="cuda") + L
    assert torch.equal(case.k[:, :, L:L + n, :], k_before[:, :, idx, :])
    assert torch.equal(case.v[:, :, :, L:L + n], v_before[:, :, :, idx])
    assert torch.equal(case.k[:, :, :L], k_before[:, :, :L])
    assert torch.equal(case.v[:, :, :, :L], v_before[:, :, :, :L])
    # restore so the case can be reused
    case.k.copy_(k_before)
    case.v.copy_(v_before)
    return n


def _check_tree_kv(case, tree, res_o, L=None):
    L = case.L if L is None else L
    T = tree.T
    for l in range(case.shape.n_layers):
        gk = O.to_f64(case.k[l, :, L:L + T, :])
        gv = O.to_f64(case.v[l, :, :, L:L + T]).transpose(0, 2, 1)
        check_logits(gk, res_o["tree_k"][l], case.shape.dtype, f"tree K layer {l}")
        check_logits(gv, res_o["tree_v"][l], case.shape.dtype, f"tree V layer {l}")


@pytest.fixture(scope="module")
def tiny_case():
    return make_case(workload("tiny"))


def test_tiny_f32_step(tiny_case):
    case = tiny_case
    ws = workspace(case, 128)
    for off in range(3):
        tree = tree_for(case, seed_offset=off)
        say(f"[tiny] T={tree.T}")
        res = gpu_step(case, tree, ws)
        ref = oracle_step(case, tree)
        check_logits(res["logits"], ref["logits"], "f32")
        check_pred(res["pred"], ref["logits"], "f32")
        _check_tree_kv(case, tree, ref)
        _accept_and_compact(case, tree, res, ws)
    assert ppd.ppd_device_status(ws) == 0


@pytest.fixture(scope="module")
def small_case():
    return make_case(workload("small"))


@pytest.mark.parametrize("spec", ["total:40", "chain:1", "total:16", "total:17", "total:64",
                                  "total:90", "total:100", "total:128"])
def test_small_bf16_tree_sizes(small_case, spec):
    case = small_case
    tree = tree_for(case, spec=spec)
    say(f"[small] {spec} T={tree.T}")
    ws = workspace(case, tree.T)
    res = gpu_step(case, tree, ws)
    ref = oracle_step(case, tree)
    check_logits(res["logits"], ref["logits"], "bf16")
    check_pred(res["pred"], ref["logits"], "bf16")
    _check_tree_kv(case, tree, ref)
    _accept_and_compact(case, tree, res, ws)
    assert ppd.ppd_device_status(ws) == 0


@pytest.mark.parametrize("L", [0, 1, 31, 32, 33, 95, 300])
def test_small_bf16_cache_lengths(small_case, L):
    """Empty and ragged prefixes: the key range [0, L + T) crosses 32-key
    blocks at every offset."""
    case = small_case
    tree = tree_for(case, spec="total:40", seed_offset=L)
    say(f"[small] L={L} T={tree.T}")
    ws = workspace(case, tree.T)
    res = gpu_step(case, tree, ws, L=L)
    ref = oracle_step(case, tree, L=L)
    check_logits(res["logits"], ref["logits"], "bf16")
    check_pred(res["pred"], ref["logits"], "bf16")


@pytest.fixture(scope="module")
def small_long_case():
    return make_case(workload("small", cache_len=2000))


@pytest.mark.parametrize("L,spec", [(2000, "total:40"), (2000, "total:128"), (700, "total:17"),
                                    (1999, "total:64")])
def test_small_bf16_long_prefix(small_long_case, L, spec):
    """Prefixes long enough for the attention to split the keys across
    workgroups (the split partials are merged by the last split)."""
    case = small_long_case
    tree = tree_for(case, spec=spec, seed_offset=L)
    say(f"[small-long] L={L} T={tree.T}")
    ws = workspace(case, tree.T)
    res = gpu_step(case, tree, ws, L=L)
    ref = oracle_step(case, tree, L=L)
    check_logits(res["logits"], ref["logits"], "bf16")
    check_pred(res["pred"], ref["logits"], "bf16")
    _check_tree_kv(case, tree, ref, L=L)


@pytest.mark.parametrize("name", ["wide", "mid", "wide-gqa"])
def test_wide_heads_and_ffn(name):
    """7B- or 1.4B-wide heads and ffn over a narrow hidden size: QKV and
    gate/up run the 3-group tiles (gate/up's last tile ragged; with 64 heads
    over 8 kv heads the last QKV tile too) or the 2-group tiles with one
    k-step per wave, every output against the oracle."""
    case = make_case(workload(name))
    for spec in ("total:40", "total:64", "total:128"):
        tree = tree_for(case, spec=spec)
        say(f"[{name}] T={tree.T}")
        ws = workspace(case, tree.T)
        res = gpu_step(case, tree, ws)
        ref = oracle_step(case, tree)
        check_logits(res["logits"], ref["logits"], "bf16")
        check_pred(res["pred"], ref["logits"], "bf16")
        _check_tree_kv(case, tree, ref)


def test_small_gqa():
    case = make_case(workload("small-gqa"))
    for spec in ("total:29", "total:70"):
        tree = tree_for(case, spec=spec)
        say(f"[gqa] T={tree.T}")
        ws = workspace(case, tree.T)
        res = gpu_step(case, tree, ws)
        ref = oracle_step(case, tree)
        check_logits(res["logits"], ref["logits"], "bf16")
        _check_tree_kv(case, tree, ref)


def test_logits_optional_and_deterministic(small_case):
    case = small_case
    tree = tree_for(case, spec="total:64")
    ws = workspace(case, tree.T)
    a = gpu_step(case, tree, ws)
    b = gpu_step(case, tree, ws, logits=False)
    c = gpu_step(case, tree, ws)
    assert np.array_equal(a["pred"], b["pred"])
    assert np.array_equal(a["logits"], c["logits"])   # bitwise: fixed reduction orders


def test_bad_token_sets_device_status(small_case):
    case = small_case
    tree = tree_for(case, spec="total:16")
    tree.ids[3] = case.shape.vocab + case.shape.n_prompt + 5
    ws = workspace(case, tree.T)
    gpu_step(case, tree, ws)
    assert ppd.ppd_device_status(ws, clear=True) & ppd.PPD_DEV_BAD_TOKEN
    assert ppd.ppd_device_status(ws) == 0


def test_tiny_multistep_lossless(tiny_case):
    """Verify -> accept -> compact on the GPU for several steps, with the
    true greedy continuation planted along a random path: the emitted tokens
    are the vanilla greedy sequence (Section 5.1: output identical to the
    original model).  Planted tokens come from the oracle."""
    case = tiny_case
    sh = case.shape
    k0, v0 = case.k.clone(), case.v.clone()
    kc, vc = O.copy_cache(case.kc_host, case.vc_host)
    L, tok = case.L, case.root
    ws = workspace(case, 128)
    rng = np.random.default_rng(3)
    emitted = []
    for s in range(5):
        tree = make_tree("candidates:10", sh.vocab, 3, 4, 900 + s, tok)
        truth = O.greedy_decode(case.oracle_model, kc, vc, L, tok, 6, "f32")
        node = int(rng.integers(1, tree.n_candidates))
        nodes = O.path_tokens(tree.parent, list(range(tree.T)), node)
        for kk, nd in enumerate(nodes[1:]):
            tree.ids[nd] = truth[kk]
        res = gpu_step(case, tree, ws, logits=False, L=L)
        tt = res["tt"]
        path = torch.zeros(tree.T, dtype=torch.int32, device="cuda")
        n_path = torch.zeros(1, dtype=torch.int32, device="cuda")
        nxt = torch.zeros(1, dtype=torch.int32, device="cuda")
        ppd.ppd_accept(tree.T, tt["parent"], tt["ids"], torch.from_numpy(res["pred"]).cuda(),
                       sh.vocab, path, n_path, nxt, ws)
        ppd.ppd_kv_compact(case.model, ppd.KVCache(case.k, case.v), L, path, n_path)
        torch.cuda.synchronize()
        n = int(n_path.item())
        assert n >= len(nodes)
        p = path[:n].cpu().tolist()
        emitted += [int(tree.ids[j]) for j in p[1:]] + [int(nxt.item())]
        say(f"[e2e] step {s}: accepted {n - 1} candidates")
        # advance the oracle's cache with the same accepted tokens
        for kk, j in enumerate(p):
            O.decode_token(case.oracle_model, kc, vc, L + kk, int(tree.ids[j]), "f32")
        L += n
        tok = int(nxt.item())
    ref = O.greedy_decode(case.oracle_model, case.kc_host, case.vc_host, case.L, case.root,
                          len(emitted), "f32")
    assert emitted == ref
    case.k.copy_(k0)
    case.v.copy_(v0)


def root_only_tree(case):
    """T = 1: the root alone, i.e. vanilla one-token decoding (reading c1)."""
    return Tree(np.array([-1], np.int32), np.array([case.root], np.int32), 1)


def vanilla_decode_reference(case, L):
    """Logits and keys / values of the root decoded alone by the oracle's
    plain decoder (no tree, no mask) on a copy of the cache."""
    sh = case.shape
    kc = [np.zeros((sh.n_kv_heads, L + 1, sh.head_dim)) for _ in range(sh.n_layers)]
    vc = [np.zeros((sh.n_kv_heads, L + 1, sh.head_dim)) for _ in range(sh.n_layers)]
    for l in range(sh.n_layers):
        kc[l][:, :L] = case.kc_host[l][:, :L]
        vc[l][:, :L] = case.vc_host[l][:, :L]
    logits = O.decode_token(case.oracle_model, kc, vc, L, case.root, sh.dtype)
    return logits, [k[:, L] for k in kc], [v[:, L] for v in vc]


@pytest.mark.parametrize("name", ["tiny", "small", "small-gqa", "wide"])
def test_root_only_tree_is_vanilla_decode(name, tiny_case, small_case):
    """A one-node tree is one step of ordinary decoding: its logits, greedy
    token and cached key / value equal the oracle's plain decoder's."""
    case = {"tiny": tiny_case, "small": small_case}.get(name) or make_case(workload(name))
    sh = case.shape
    tree = root_only_tree(case)
    say(f"[root-only] {name} L={case.L}")
    ws = workspace(case, 1)
    res = gpu_step(case, tree, ws)
    ref, k_ref, v_ref = vanilla_decode_reference(case, case.L)
    check_logits(res["logits"], ref[None, :], sh.dtype, "root logits")
    check_pred(res["pred"], ref[None, :], sh.dtype)
    L = case.L
    for l in range(sh.n_layers):
        check_logits(O.to_f64(case.k[l, :, L, :]), k_ref[l], sh.dtype, f"root K layer {l}")
        check_logits(O.to_f64(case.v[l, :, :, L]), v_ref[l], sh.dtype, f"root V layer {l}")
    n = _accept_and_compact(case, tree, res, ws)
    assert n == 1
    assert ppd.ppd_device_status(ws) == 0


def _expected_packing(w, kind):
    """The packed layout of include/ppd.h, written out with numpy indexing:
    item (group, chunk, q, s, lane) = row r(group, q, lane % 16), columns
    64 chunk + 32 s + 8 (lane // 16) .. + 7; zeros past the matrix.  A group
    is 16 rows (gate/up: 16 features: q = 0 their gate rows, q = 1 their up
    rows); a QKV group holds dims 8 (g % 8) .. + 7 of head part g // 8 in
    rows 0..7 and their RoPE partners (+64) in rows 8..15."""
    rows, cols = w.shape
    kc = cols // 64
    r = np.arange(16)
    if kind == ppd.PPD_W_GATE_UP:
        F = rows // 2
        G, S = -(-F // 16), 2
        f = 16 * np.arange(G)[:, None] + r[None, :]                  # [G][16]
        tr = np.stack([np.where(f < F, f, rows), np.where(f < F, F + f, rows)], axis=1)
    elif kind == ppd.PPD_W_QKV:
        G, S = rows // 16, 1
        g = np.arange(G)[:, None]
        tr = (128 * (g // 8) + np.where(r < 8, 0, 64)[None, :] + 8 * (g % 8) + (r % 8)[None, :])[:, None, :]
    else:
        G, S = -(-rows // 16), 1
        tr = (16 * np.arange(G)[:, None] + r[None, :])[:, None, :]
        tr = np.where(tr < rows, tr, rows)
    wp = np.zeros((rows + 1, cols), dtype=w.dtype)               # row `rows`: zeros
    wp[:rows] = w
    lane = np.arange(64)
    out = np.zeros((G, kc, S, 2, 64, 8), dtype=w.dtype)
    for q in range(S):
        rr = tr[:, q, lane % 16]                                  # [G][64]
        for s in range(2):
            for c in range(kc):
                col = 64 * c + 32 * s + 8 * (lane // 16)
                idx = col[:, None] + np.arange(8)[None, :]        # [64][8]
                out[:, c, q, s] = wp[rr[:, :, None], idx[None, :, :]]
    return out


@pytest.mark.parametrize("kind,rows,cols", [(ppd.PPD_W_LM_HEAD, 1000, 512),
                                            (ppd.PPD_W_GATE_UP, 2 * 1344, 512),
                                            (ppd.PPD_W_DOWN, 512, 1344),
                                            (ppd.PPD_W_QKV, 6 * 128, 256),
                                            (ppd.PPD_W_GATE_UP, 2 * 11008, 512),
                                            (ppd.PPD_W_QKV, 96 * 128, 512),
                                            (ppd.PPD_W_QKV, 96 * 128, 256),
                                            (ppd.PPD_W_QKV, 48 * 128, 512),
                                            (ppd.PPD_W_QKV, 80 * 128, 512),
                                            (ppd.PPD_W_GATE_UP, 2 * 5632, 512)])
def test_pack_weight_layout(kind, rows, cols):
    say(f"[pack] kind={kind} {rows}x{cols}")
    g = torch.Generator().manual_seed(rows * 7 + cols)
    w = torch.randint(0, 1 << 16, (rows, cols), generator=g, dtype=torch.int32)
    w = (w & 0x7F7F).to(torch.int16)                    # finite bf16 bit patterns
    src = w.view(torch.bfloat16).cuda()
    packed = ppd.ppd_pack_weight(kind, src)
    torch.cuda.synchronize()
    got = packed.cpu().view(torch.int16).numpy()
    exp = _expected_packing(w.numpy(), kind).reshape(-1)
    assert got.shape == exp.shape
    assert np.array_equal(got, exp)
