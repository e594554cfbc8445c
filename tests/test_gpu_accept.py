"""Device acceptance and KV compaction on injected greedy tokens (Section 3:
exact matching; Section 5.3: one KV cache, only accepted tokens committed).

The greedy tokens are not produced by a model here: they are written into
`pred` directly, so that the acceptance kernel sees every situation exact
matching can meet -- long accepted chains, several verified branches of equal
depth (duplicate sibling tokens: the smallest node index wins), accepted nodes
past index 64, prompt nodes on and off the matching paths, a root alone --
and is compared bit for bit with the oracle's `accept` and with a brute-force
enumeration written here.  Compaction is then checked row for row on deep
paths, and against a count larger than the path buffer (clamped on the
device)."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2405_18628_amd as ppd
from gpu_cases import say
from synth.configs import ModelShape

pytestmark = pytest.mark.gpu

VOCAB = 40     # small, so that random greedy tokens match often
N_PROMPT = 3


def _random_tree(rng, T, style):
    """Topological parent array and ids of T nodes.  style: "random"
    (parent uniform over earlier nodes), "deep" (mostly the previous node),
    "bushy" (parent among the first few nodes)."""
    parent = np.full(T, -1, np.int32)
    for i in range(1, T):
        if style == "deep":
            parent[i] = i - 1 if rng.random() < 0.8 else rng.integers(0, i)
        elif style == "bushy":
            parent[i] = rng.integers(0, min(i, 6))
        else:
            parent[i] = rng.integers(0, i)
    ids = rng.integers(0, VOCAB, T).astype(np.int32)
    # prompt ids: a few nodes (15 %, 2 % in deep trees, so that long chains
    # stay candidates), and then (as the ABI asks) their whole subtrees
    p_prompt = 0.02 if style == "deep" else 0.15
    is_prompt = np.zeros(T, bool)
    for i in range(1, T):
        is_prompt[i] = is_prompt[parent[i]] or rng.random() < p_prompt
    ids[is_prompt] = VOCAB + rng.integers(0, N_PROMPT, int(is_prompt.sum()))
    ids[0] = rng.integers(0, VOCAB)
    return parent, ids


def _plant(rng, parent, ids, pred, target):
    """Make every vocabulary node on target's root path match its parent's
    greedy token (stops at a prompt node, which can never match)."""
    path = []
    j = int(target)
    while j > 0:
        path.append(j)
        j = int(parent[j])
    for j in reversed(path):
        if ids[j] >= VOCAB:
            break
        pred[parent[j]] = ids[j]


def _duplicate_siblings(rng, parent, ids, n):
    """Give n random nodes the token of an earlier sibling (equal-depth
    verified branches when that token is the parent's greedy token)."""
    T = len(parent)
    for _ in range(n):
        i = int(rng.integers(1, T))
        sib = [j for j in range(1, i) if parent[j] == parent[i] and ids[j] < VOCAB]
        if sib and ids[i] < VOCAB:
            ids[i] = ids[sib[int(rng.integers(0, len(sib)))]]


def _brute_accept(parent, ids, pred):
    """Every node's root path checked directly; the deepest verified node,
    ties to the smallest index."""
    T = len(parent)
    best, best_depth = 0, 0
    for i in range(T):
        path = []
        j = i
        while j != -1:
            path.append(j)
            j = int(parent[j])
        path.reverse()
        ok = all(0 <= ids[c] < VOCAB and ids[c] == pred[parent[c]] for c in path[1:])
        if ok and len(path) - 1 > best_depth:
            best, best_depth = i, len(path) - 1
    path = []
    j = best
    while j != -1:
        path.append(j)
        j = int(parent[j])
    return path[::-1], best_depth + 1, int(pred[best])


def _cases(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for c in range(n):
        T = int(rng.choice([1, 2, 3, 7, 40, 63, 64, 65, 100, 127, 128, int(rng.integers(1, 129))]))
        style = ("random", "deep", "bushy")[c % 3]
        parent, ids = _random_tree(rng, T, style)
        pred = rng.integers(0, VOCAB + 5, T).astype(np.int32)  # some greedy tokens out of vocab
        if T > 1:
            _duplicate_siblings(rng, parent, ids, int(rng.integers(0, 4)))
            # plant a path to a random node; for large trees often past index 64
            lo = 64 if (T > 64 and rng.random() < 0.6) else 1
            _plant(rng, parent, ids, pred, int(rng.integers(lo, T)))
            if rng.random() < 0.3:  # and a second, competing one
                _plant(rng, parent, ids, pred, int(rng.integers(1, T)))
        out.append((parent, ids, pred))
    return out


def test_accept_injected_tokens_bit_exact():
    cases = _cases(600, seed=12345)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
    ws = torch.zeros(256, dtype=torch.uint8, device="cuda")
    ppd.ppd_workspace_init(ws)
    outs = []
    for parent, ids, pred in cases:
        T = len(parent)
        path = torch.full((T,), -7, dtype=torch.int32, device="cuda")
        n_path = torch.full((1,), -7, dtype=torch.int32, device="cuda")
        nxt = torch.full((1,), -7, dtype=torch.int32, device="cuda")
        ins = (dev(parent), dev(ids), dev(pred))
        ppd.ppd_accept(T, ins[0], ins[1], ins[2], VOCAB, path, n_path, nxt, ws)
        outs.append((ins, path, n_path, nxt))
    torch.cuda.synchronize()
    assert ppd.ppd_device_status(ws) == 0
    stats = {"deep": 0, "past64": 0, "ties": 0}
    for (parent, ids, pred), (_, path, n_path, nxt) in zip(cases, outs):
        opath, on, onext = O.accept(parent, ids, pred, VOCAB)
        bpath, bn, bnext = _brute_accept(parent, ids, pred)
        assert (list(opath), on, onext) == (bpath, bn, bnext)
        n = int(n_path.item())
        assert n == on and int(nxt.item()) == onext
        assert path[:n].cpu().tolist() == list(opath)
        stats["deep"] += on >= 4
        stats["past64"] += int(opath[-1]) >= 64
        # equally deep verified nodes other than the chosen one
        depth, _ = O.build_mask(parent)
        ok = np.zeros(len(parent), bool)
        ok[0] = True
        for i in range(1, len(parent)):
            ok[i] = ok[parent[i]] and ids[i] < VOCAB and ids[i] == pred[parent[i]]
        stats["ties"] += int(np.sum(ok & (depth == on - 1))) > 1
    say(f"  accept cases: {len(cases)}, paths >= 4 tokens {stats['deep']}, accepted node "
        f">= 64: {stats['past64']}, equal-depth ties: {stats['ties']}")
    assert stats["deep"] > 50 and stats["past64"] > 30 and stats["ties"] > 10


def test_accept_bad_parent_sets_status_bit():
    """A parent array outside the contract (not topological, root not -1)
    sets PPD_DEV_BAD_PARENT; the kernel still ends and writes a path within
    the tree."""
    ws = torch.zeros(256, dtype=torch.uint8, device="cuda")
    for parent in ([0, 0, 1, 2], [-1, 0, 5, 1], [-1, 1, 0, 0], [-1, 0, -3, 2]):
        ppd.ppd_workspace_init(ws)
        T = len(parent)
        par = torch.tensor(parent, dtype=torch.int32, device="cuda")
        ids = torch.tensor([1, 2, 3, 4], dtype=torch.int32, device="cuda")
        pred = torch.tensor([2, 3, 4, 5], dtype=torch.int32, device="cuda")
        path = torch.full((T,), -7, dtype=torch.int32, device="cuda")
        n_path = torch.zeros(1, dtype=torch.int32, device="cuda")
        nxt = torch.zeros(1, dtype=torch.int32, device="cuda")
        ppd.ppd_accept(T, par, ids, pred, VOCAB, path, n_path, nxt, ws)
        torch.cuda.synchronize()
        st = ppd.ppd_device_status(ws)
        assert st & ppd.PPD_DEV_BAD_PARENT, parent
        n = int(n_path.item())
        assert 1 <= n <= T
        assert all(0 <= int(x) < T for x in path[:n].cpu().tolist())


def test_accept_root_only():
    """T = 1: vanilla decoding -- the root is the whole path, the bonus token
    is its greedy token."""
    ws = torch.zeros(256, dtype=torch.uint8, device="cuda")
    ppd.ppd_workspace_init(ws)
    par = torch.tensor([-1], dtype=torch.int32, device="cuda")
    ids = torch.tensor([7], dtype=torch.int32, device="cuda")
    pred = torch.tensor([11], dtype=torch.int32, device="cuda")
    path = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    n_path = torch.zeros(1, dtype=torch.int32, device="cuda")
    nxt = torch.zeros(1, dtype=torch.int32, device="cuda")
    ppd.ppd_accept(1, par, ids, pred, VOCAB, path, n_path, nxt, ws)
    torch.cuda.synchronize()
    assert path.tolist() == [0] and int(n_path.item()) == 1 and int(nxt.item()) == 11
    assert ppd.ppd_device_status(ws) == 0


# ---------------------------------------------------------------------------
# compaction of deep paths

SHAPE = ModelShape("compact-bf16", 3, 256, 4, 2, 128, 256, VOCAB, "bf16")


def _model_desc(shape, dev_tensors):
    """A model description whose weights are never read by ppd_kv_compact
    (it needs only the layer / head counts and the dtype)."""
    z = lambda *s: torch.zeros(*s, dtype=torch.bfloat16, device="cuda")
    H = shape.hidden
    lay = {"attn_norm": z(H), "w_qkv": z(shape.qkv_rows, H),
           "w_o": z(H, shape.n_heads * shape.head_dim),
           "mlp_norm": z(H), "w_gate_up": z(2 * shape.ffn, H), "w_down": z(H, shape.ffn)}
    W = {"tok_emb": z(shape.vocab, H), "prompt_emb": z(shape.n_prompt, H), "final_norm": z(H),
         "lm_head": z(shape.vocab, H), "layers": [lay] * shape.n_layers}
    dev_tensors.append(W)
    return ppd.Model(shape, W)


@pytest.mark.parametrize("L,cap", [(0, 136), (37, 168), (300, 432), (1000, 1128)])
def test_compact_deep_paths_bit_exact(L, cap):
    keep = []
    model = _model_desc(SHAPE, keep)
    rng = np.random.default_rng(L)
    g = torch.Generator(device="cuda")
    g.manual_seed(L + 1)
    nl, nkv, d = SHAPE.n_layers, SHAPE.n_kv_heads, SHAPE.head_dim
    k = torch.randn((nl, nkv, cap, d), generator=g, device="cuda").to(torch.bfloat16)
    v = torch.randn((nl, nkv, d, cap), generator=g, device="cuda").to(torch.bfloat16)
    ws = torch.zeros(256, dtype=torch.uint8, device="cuda")
    ppd.ppd_workspace_init(ws)
    for trial in range(6):
        T = int(min(cap - L, rng.choice([1, 9, 64, 65, 128])))
        parent, ids = _random_tree(rng, T, "deep")
        ids[ids >= VOCAB] = ids[ids >= VOCAB] % VOCAB  # all candidates: long paths possible
        pred = rng.integers(0, VOCAB, T).astype(np.int32)
        if T > 1:
            _plant(rng, parent, ids, pred, T - 1 if trial % 2 else int(rng.integers(1, T)))
        opath, on, _ = O.accept(parent, ids, pred, VOCAB)
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
        path = torch.zeros(T, dtype=torch.int32, device="cuda")
        n_path = torch.zeros(1, dtype=torch.int32, device="cuda")
        nxt = torch.zeros(1, dtype=torch.int32, device="cuda")
        ppd.ppd_accept(T, dev(parent), dev(ids), dev(pred), VOCAB, path, n_path, nxt, ws)
        k0, v0 = k.clone(), v.clone()
        len_dev = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        ppd.ppd_kv_compact(model, ppd.KVCache(k, v, len_dev), L, path, n_path)
        torch.cuda.synchronize()
        assert int(n_path.item()) == on and int(len_dev.item()) == L + on
        # the oracle's commit on exact float64 copies of the bf16 rows
        kc = [O.to_f64(k0[l]) for l in range(nl)]
        vc = [O.to_f64(v0[l]).transpose(0, 2, 1).copy() for l in range(nl)]
        tk = [O.to_f64(k0[l, :, L:L + T, :]) for l in range(nl)]
        tv = [O.to_f64(v0[l, :, :, L:L + T]).transpose(0, 2, 1) for l in range(nl)]
        O.kv_compact(kc, vc, tk, tv, L, opath)
        for l in range(nl):
            assert np.array_equal(O.to_f64(k[l]), kc[l])
            assert np.array_equal(O.to_f64(v[l]).transpose(0, 2, 1), vc[l])
        say(f"  L={L} T={T} n_path={on}")
    assert ppd.ppd_device_status(ws) == 0


def test_compact_clamps_count_to_path_length():
    """A count larger than the path buffer (stale or foreign) moves only
    path_len rows: the device clamps it."""
    keep = []
    model = _model_desc(SHAPE, keep)
    L, cap = 16, 176
    g = torch.Generator(device="cuda")
    g.manual_seed(3)
    nl, nkv, d = SHAPE.n_layers, SHAPE.n_kv_heads, SHAPE.head_dim
    k = torch.randn((nl, nkv, cap, d), generator=g, device="cuda").to(torch.bfloat16)
    v = torch.randn((nl, nkv, d, cap), generator=g, device="cuda").to(torch.bfloat16)
    k0, v0 = k.clone(), v.clone()
    path = torch.tensor([0, 5, 9], dtype=torch.int32, device="cuda")
    n_path = torch.tensor([100], dtype=torch.int32, device="cuda")
    len_dev = torch.zeros(1, dtype=torch.int32, device="cuda")
    ppd.ppd_kv_compact(model, ppd.KVCache(k, v, len_dev), L, path, n_path)
    torch.cuda.synchronize()
    assert int(len_dev.item()) == L + 3
    idx = torch.tensor([L, L + 5, L + 9], device="cuda")
    assert torch.equal(k[:, :, L:L + 3], k0[:, :, idx])
    assert torch.equal(v[:, :, :, L:L + 3], v0[:, :, :, idx])
    assert torch.equal(k[:, :, L + 3:], k0[:, :, L + 3:])
    assert torch.equal(v[:, :, :, L + 3:], v0[:, :, :, L + 3:])
    assert torch.equal(k[:, :, :L], k0[:, :, :L])


def test_read_probe_reads_every_byte():
    """The HBM read probe (the measurement aid behind bench.py
    --stream-ceiling) reads the whole buffer: its XOR sink equals the XOR of
    every 32-bit word, for sizes that leave ragged pieces."""
    rng = np.random.default_rng(5)
    for n_words in (4, 4 * 1000, 4 * 65537, 4 * (1 << 20) + 12):
        host = rng.integers(0, 2 ** 32, size=n_words, dtype=np.uint64).astype(np.uint32)
        buf = torch.from_numpy(host.view(np.int32)).cuda()
        sink = torch.zeros(1, dtype=torch.int32, device="cuda")
        ppd.ppd_read_probe(buf, sink)
        torch.cuda.synchronize()
        want = np.bitwise_xor.reduce(host)
        assert np.uint32(sink.cpu().numpy().view(np.uint32)[0]) == want, n_words
