"""Pins of the CPU oracle against things other than itself.

* HuggingFace Llama (a library implementation) driven by a custom 4-D mask and
  position ids reproduces the oracle's tree logits and prefill cache.
* Brute force: every tree node's logits equal an ordinary token-by-token
  causal decode of its root-to-node path (Section 4.1: ancestors-only
  attention; Section 3.1: prompt tokens at the positions of the tokens they
  stand for).
* Special cases: a chain tree is causal multi-token decoding; a one-node tree
  is vanilla one-token decoding (Table 1: vanilla tau = 1.00).
* Invariants: non-ancestor nodes do not influence a node; relabelling nodes
  permutes rows.
* Closed forms for RMSNorm, rotary embedding, SiLU, softmax, bf16 rounding.
* Acceptance: brute-force enumeration of root paths; Proposition 1's expected
  accept length by Monte Carlo; multi-step losslessness (Section 5.1: greedy
  output is identical to the original model's).
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle as O
from synth import workload
from synth.configs import ModelShape
from synth.model import make_weights, tokens
from synth.trees import make_tree, tree_from_parents

GOLD = os.path.join(os.path.dirname(__file__), "golden")

MICRO = ModelShape("micro", 2, 64, 4, 2, 16, 96, 50, "f32")


def _setup(w, gain_std=0.1, store="f32", L=None, shape=None):
    sh = shape or w.shape
    W = make_weights(sh, w.seeds["weights"], gain_std=gain_std)
    m = O.Model(sh, W)
    L = w.cache_len if L is None else L
    ids = tokens(L + 1, sh.vocab, w.seeds["tokens"]).numpy()
    kc, vc, _ = O.prefill(m, ids[:-1], L + 160, store)
    return sh, W, m, kc, vc, L, int(ids[-1])


@pytest.fixture(scope="module")
def tiny():
    return _setup(workload("tiny"))


# ---------------------------------------------------------------- library pin

def test_matches_hf_llama_tree_forward():
    from hf_reference import build_hf_llama, hf_prefill, hf_tree_logits
    w = workload("tiny", cache_len=48)
    sh, W, m, kc, vc, L, root = _setup(w, store=None)
    hf = build_hf_llama(sh, W)
    ids = tokens(L + 1, sh.vocab, w.seeds["tokens"]).numpy()
    hf_logits, pkv = hf_prefill(hf, ids[:-1])
    k_hf = pkv.layers[1].keys[0].numpy()
    v_hf = pkv.layers[1].values[0].numpy()
    # the prefill's last logits: the oracle's plain decoder (decode_token)
    # against the library's causal forward
    _, _, last = O.prefill(m, ids[:-1], L + 8, None)
    assert np.abs(np.asarray(hf_logits)[-1, :sh.vocab] - last).max() < 2e-5
    assert np.abs(k_hf - kc[1][:, :L]).max() < 1e-5
    assert np.abs(v_hf - vc[1][:, :L]).max() < 1e-5
    for seed in range(3):
        tree = make_tree("candidates:10", sh.vocab, 3, 4, 77 + seed, root)
        res = O.verify_forward(m, kc, vc, L, tree.ids, tree.parent, None)
        depth, anc = O.build_mask(tree.parent)
        ref = hf_tree_logits(hf, pkv, L, tree.ids, depth, anc, sh.vocab)
        assert np.abs(ref - res["logits"]).max() < 2e-5


def test_matches_hf_llama_gqa():
    from hf_reference import build_hf_llama, hf_prefill, hf_tree_logits
    w = workload("small-gqa")
    sh = MICRO
    W = make_weights(sh, 5, gain_std=0.2)
    m = O.Model(sh, W)
    ids = tokens(21, sh.vocab, 6).numpy()
    kc, vc, _ = O.prefill(m, ids[:-1], 64, None)
    hf = build_hf_llama(sh, W)
    _, pkv = hf_prefill(hf, ids[:-1])
    tree = make_tree("total:17", sh.vocab, 3, 3, 9, int(ids[-1]))
    res = O.verify_forward(m, kc, vc, 20, tree.ids, tree.parent, None)
    depth, anc = O.build_mask(tree.parent)
    ref = hf_tree_logits(hf, pkv, 20, tree.ids, depth, anc, sh.vocab)
    assert np.abs(ref - res["logits"]).max() < 1e-5


# ---------------------------------------------------------------- brute force

@pytest.mark.parametrize("spec,seed", [("candidates:10", 1), ("candidates:10", 2), ("total:25", 3)])
def test_tree_nodes_equal_causal_paths(tiny, spec, seed):
    sh, W, m, kc, vc, L, root = tiny
    tree = make_tree(spec, sh.vocab, 3, 4, seed, root)
    res = O.verify_forward(m, kc, vc, L, tree.ids, tree.parent, "f32")
    for i in range(tree.T):
        seq = O.path_tokens(tree.parent, tree.ids, i)
        ref = O.causal_logits(m, kc, vc, L, seq, "f32")[-1]
        assert np.abs(ref - res["logits"][i]).max() < 1e-9


def test_tree_nodes_equal_causal_paths_bf16():
    w = workload("small", n_layers=1, cache_len=40)
    sh, W, m, kc, vc, L, root = _setup(w, store="bf16")
    tree = make_tree("total:20", sh.vocab, 3, 4, 5, root)
    res = O.verify_forward(m, kc, vc, L, tree.ids, tree.parent, "bf16")
    for i in range(tree.T):
        seq = O.path_tokens(tree.parent, tree.ids, i)
        ref = O.causal_logits(m, kc, vc, L, seq, "bf16")[-1]
        assert np.abs(ref - res["logits"][i]).max() < 1e-9


def test_depth_taps_are_the_cut_models(tiny):
    """tap_logits[n]: the logits of the same model cut to its first n layers
    (its own forward, run separately)."""
    sh, W, m, kc, vc, L, root = tiny
    tree = make_tree("candidates:10", sh.vocab, 3, 4, 4, root)
    res = O.verify_forward(m, kc, vc, L, tree.ids, tree.parent, "f32", taps=(1, 2))
    W1 = dict(W)
    W1["layers"] = W["layers"][:1]
    m1 = O.Model(sh.with_layers(1), W1)
    cut = O.verify_forward(m1, kc[:1], vc[:1], L, tree.ids, tree.parent, "f32")
    assert np.array_equal(res["tap_logits"][1], cut["logits"])
    assert np.array_equal(res["tap_logits"][2], res["logits"])


def test_float32_sums_agree_at_float32_precision(tiny):
    """acc="f32" computes the same values with float32 products and residual:
    within the float32 tolerance of the float64 sums, and not identical."""
    sh, W, m, kc, vc, L, root = tiny
    tree = make_tree("total:25", sh.vocab, 3, 4, 6, root)
    a = O.verify_forward(m, kc, vc, L, tree.ids, tree.parent, "f32")
    b = O.verify_forward(m, kc, vc, L, tree.ids, tree.parent, "f32", acc="f32")
    err = np.abs(a["logits"] - b["logits"])
    assert err.max() < 1e-4 * (1 + np.abs(a["logits"]).max())
    assert err.max() > 0


def test_chain_tree_is_multitoken_decode(tiny):
    sh, W, m, kc, vc, L, root = tiny
    seq = [root] + list(tokens(5, sh.vocab, 99).numpy()) + [sh.vocab + j for j in range(3)]
    parent = [-1] + list(range(len(seq) - 1))
    res = O.verify_forward(m, kc, vc, L, seq, parent, "f32")
    ref = O.causal_logits(m, kc, vc, L, seq, "f32")
    assert np.abs(ref - res["logits"]).max() < 1e-9
    # and the tree keys are the keys a causal decode would cache
    kc2, vc2 = O.copy_cache(kc, vc)
    for j, t in enumerate(seq):
        O.decode_token(m, kc2, vc2, L + j, t, "f32")
    for l in range(sh.n_layers):
        assert np.abs(kc2[l][:, L:L + len(seq)] - res["tree_k"][l]).max() < 1e-12
        assert np.abs(vc2[l][:, L:L + len(seq)] - res["tree_v"][l]).max() < 1e-12


def test_single_node_tree_is_vanilla_decode(tiny):
    sh, W, m, kc, vc, L, root = tiny
    res = O.verify_forward(m, kc, vc, L, [root], [-1], "f32")
    kc2, vc2 = O.copy_cache(kc, vc)
    ref = O.decode_token(m, kc2, vc2, L, root, "f32")
    assert np.abs(ref - res["logits"][0]).max() < 1e-12
    path, n_path, nxt = O.accept([-1], [root], O.argmax_first(res["logits"]), sh.vocab)
    assert n_path == 1 and list(path) == [0] and nxt == int(np.argmax(ref))


# ---------------------------------------------------------------- invariants

def test_non_ancestors_do_not_matter(tiny):
    sh, W, m, kc, vc, L, root = tiny
    tree = make_tree("candidates:10", sh.vocab, 3, 4, 11, root)
    full = O.verify_forward(m, kc, vc, L, tree.ids, tree.parent, "f32")["logits"]
    # keep only the ancestor closure of one deep node
    depth, anc = O.build_mask(tree.parent)
    target = int(np.argmax(depth))
    keep = [j for j in range(tree.T) if anc[target, j]]
    remap = {old: new for new, old in enumerate(keep)}
    sub_parent = [-1 if tree.parent[j] < 0 else remap[int(tree.parent[j])] for j in keep]
    sub = O.verify_forward(m, kc, vc, L, tree.ids[keep], sub_parent, "f32")["logits"]
    for new, old in enumerate(keep):
        assert np.abs(sub[new] - full[old]).max() < 1e-12


def test_relabel_permutes_rows(tiny):
    sh, W, m, kc, vc, L, root = tiny
    tree = make_tree("candidates:10", sh.vocab, 3, 4, 12, root)
    res = O.verify_forward(m, kc, vc, L, tree.ids, tree.parent, "f32")["logits"]
    # another topological order: depth-first
    children = {i: [] for i in range(tree.T)}
    for i in range(1, tree.T):
        children[int(tree.parent[i])].append(i)
    order, stack = [], [0]
    while stack:
        j = stack.pop()
        order.append(j)
        stack.extend(reversed(children[j]))
    new_of = {old: new for new, old in enumerate(order)}
    par2 = [-1] + [new_of[int(tree.parent[o])] for o in order[1:]]
    res2 = O.verify_forward(m, kc, vc, L, tree.ids[order], par2, "f32")["logits"]
    assert np.abs(res2 - res[order]).max() < 1e-12


# ---------------------------------------------------------------- closed forms

def test_rmsnorm_closed_form():
    x = np.array([[3.0, -4.0], [1.0, 1.0]])
    r = O.rms_scale(x, 0.0)
    assert np.allclose(r, [1 / math.sqrt(12.5), 1.0])
    c = 0.37
    r = O.rms_scale(np.full((1, 8), c), 1e-6)
    assert abs(r[0] - 1 / math.sqrt(c * c + 1e-6)) < 1e-15
    a, r = O.normed_rows(np.array([[2.0, 0.0, -2.0, 0.0]]), np.array([1.0, 2.0, 3.0, 4.0]), 0.0, None)
    assert np.allclose(r[:, None] * a, [[math.sqrt(2), 0, -3 * math.sqrt(2), 0]])


def test_rope_is_a_rotation_by_pos_times_frequency():
    d, base = 8, 100.0
    pos = np.array([0, 1, 5, 1234])
    cos, sin = O.rope_tables(pos, d, base)
    x = np.random.default_rng(0).standard_normal((4, 1, d))
    y = O.apply_rope(x, cos, sin)
    for n in range(4):
        for i in range(d // 2):
            th = pos[n] * base ** (-2 * i / d)
            R = np.array([[math.cos(th), -math.sin(th)], [math.sin(th), math.cos(th)]])
            ref = R @ np.array([x[n, 0, i], x[n, 0, i + d // 2]])
            assert np.allclose([y[n, 0, i], y[n, 0, i + d // 2]], ref, atol=1e-12)
    assert np.allclose(y[0], x[0])                          # position 0: identity
    # relative property: <rope(q,m), rope(k,n)> depends on m - n only
    q = np.random.default_rng(1).standard_normal((1, 1, d))
    k = np.random.default_rng(2).standard_normal((1, 1, d))

    def dot(m, n):
        cm, sm = O.rope_tables(np.array([m]), d, base)
        cn, sn = O.rope_tables(np.array([n]), d, base)
        return float(np.sum(O.apply_rope(q, cm, sm) * O.apply_rope(k, cn, sn)))
    assert abs(dot(10, 3) - dot(107, 100)) < 1e-10


def test_silu_softmax_library():
    from scipy.special import expit, softmax
    x = np.linspace(-30, 30, 101)
    assert np.allclose(O.silu(x), x * expit(x), rtol=1e-14, atol=1e-300)
    s = np.random.default_rng(3).standard_normal((4, 9)) * 5
    s[1, 3] = -np.inf
    assert np.allclose(O.softmax_rows(s), softmax(s, axis=-1), rtol=1e-14)


def test_bf16_rounding_matches_torch_and_ties_to_even():
    rng = np.random.default_rng(4)
    x = np.concatenate([rng.standard_normal(10000) * 10.0 ** rng.integers(-20, 20, 10000),
                        [0.0, -0.0, 1e-40, 3.0e38, -3.4e38]])
    ref = torch.tensor(x.astype(np.float32)).to(torch.bfloat16).double().numpy()
    assert np.array_equal(O.round_store(x, "bf16"), ref)
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties to even (1.0)
    assert O.round_store(np.array([1 + 2 ** -8]), "bf16")[0] == 1.0
    assert O.round_store(np.array([1 + 3 * 2 ** -8]), "bf16")[0] == 1 + 2 ** -6
    assert O.round_store(np.array([0.1]), "f32")[0] == float(np.float32(0.1))


def test_masks():
    parent = [-1, 0, 0, 1, 3, 2, 4]
    depth, anc = O.build_mask(parent)
    assert list(depth) == [0, 1, 1, 2, 3, 2, 4]
    assert anc[6].tolist() == [True, True, False, True, True, False, True]
    packed = O.pack_mask(anc)
    assert int(packed[6, 0]) == (1 << 0) | (1 << 1) | (1 << 3) | (1 << 4) | (1 << 6)
    chain = [-1] + list(range(99))
    d2, a2 = O.build_mask(chain)
    assert list(d2) == list(range(100))
    p2 = O.pack_mask(a2)
    assert int(p2[99, 0]) == (1 << 64) - 1 and int(p2[99, 1]) == (1 << 36) - 1
    for bad in ([0], [-1, 1], [-1, 0, 3], [-1, -1]):
        with pytest.raises(ValueError):
            O.build_mask(bad)


# ---------------------------------------------------------------- acceptance

def _brute_accept(parent, ids, pred, vocab):
    """Enumerate every root path; keep the longest whose every candidate
    matches the greedy token of its predecessor (ties: smallest end node)."""
    best = (0, [0])
    for node in range(len(parent)):
        path, j = [], node
        while j != -1:
            path.append(j)
            j = parent[j]
        path = path[::-1]
        good = all(0 <= ids[path[k]] < vocab and ids[path[k]] == pred[path[k - 1]]
                   for k in range(1, len(path)))
        if good and len(path) > len(best[1]):
            best = (node, path)
    return best[1], pred[best[0]]


def test_accept_brute_force():
    V = 7
    rng = np.random.default_rng(5)
    for trial in range(600):
        spec = ["candidates:6", "total:20", "candidates:12"][trial % 3]
        tree = make_tree(spec, V, 2, 4, 1000 + trial, int(rng.integers(V)))
        ids = tree.ids.copy()
        if trial % 4 == 3:
            # duplicate sibling tokens (allowed by the interface): equally deep
            # verified nodes can then exist and the smallest index must win
            ids[1:tree.n_candidates] = rng.integers(2, size=tree.n_candidates - 1)
        # predictions may even name prompt ids: prompt nodes still never verify
        pred = rng.integers(V + 2, size=tree.T)
        if trial % 2:
            node = int(rng.integers(tree.n_candidates))
            p = O.path_tokens(tree.parent, list(range(tree.T)), node)
            for a, b in zip(p[:-1], p[1:]):
                pred[a] = ids[b]
        if trial % 5 == 0:
            pred[:] = ids[np.maximum(np.arange(tree.T), 1)]   # prompt ids predicted too
        path, n_path, nxt = O.accept(tree.parent, ids, pred, V)
        bpath, bnxt = _brute_accept(list(tree.parent), list(ids), list(pred), V)
        assert list(path) == bpath and n_path == len(bpath) and nxt == bnxt


def test_vanilla_tau_is_one_and_table1_accounting():
    """Table 1: vanilla decoding has tau = 1.00 and throughput ~= tau / L_fp."""
    g = json.load(open(os.path.join(GOLD, "table1.json")))
    for row in g["rows"]:
        assert abs(row["tau"] / row["L_fp"] - row["T"]) / row["T"] < 0.05, row
        if row["method"] == "vanilla":
            assert row["tau"] == 1.0
    # the oracle's accounting reproduces tau = 1 for a root-only tree
    _, n_path, _ = O.accept([-1], [3], [5], 10)
    assert n_path == 1


def test_prompt_table_share_matches_table1():
    """P_tr (Table 1): 3 prompt embeddings of size hidden over the model's
    parameters reproduces 4.50e-4 % (MobileLLaMA) and 1.82e-4 % (Vicuna-7B)."""
    g = json.load(open(os.path.join(GOLD, "table1.json")))
    share = {r["model"]: r["P_tr_pct"] for r in g["rows"] if "P_tr_pct" in r}
    for name, key in (("1.4b", "MobileLLaMA"), ("7b", "Vicuna-7B")):
        sh = workload(name).shape
        pct = 100.0 * g["prompt_tokens"] * g["ept"] * sh.hidden / sh.total_params()
        assert abs(pct - share[key]) / share[key] < 0.01, (name, pct)


def test_proposition1_expected_accept_length():
    """Proposition 1: with independent acceptance probability p_d at depth d,
    the expected number of accepted candidates is the sum over candidates v of
    the product of p along the root path of v."""
    V = 4
    tree = make_tree("candidates:9", V, 3, 3, 21, 0)
    depth, anc = O.build_mask(tree.parent)
    p = {1: 0.6, 2: 0.45, 3: 0.3}
    rng = np.random.default_rng(6)
    n = 20000
    acc = 0
    cand = range(1, tree.n_candidates)
    # each node's children hold distinct tokens; the true next token after node
    # u is child c's token with prob q(c) = p_depth(c) / n_children(u), else a
    # token no child holds.
    kids = {u: [c for c in cand if tree.parent[c] == u] for u in range(tree.n_candidates)}
    q = {c: p[int(depth[c])] / len(kids[int(tree.parent[c])]) for c in cand}
    expected = sum(np.prod([q[u] for u in range(1, tree.n_candidates) if anc[v, u]]) for v in cand)
    for _ in range(n):
        pred = np.full(tree.T, V + 100)  # "no child" token (never a candidate id)
        for u in range(tree.n_candidates):
            if kids[u]:
                r = rng.random()
                c0 = 0.0
                for c in kids[u]:
                    c0 += q[c]
                    if r < c0:
                        pred[u] = tree.ids[c]
                        break
        _, n_path, _ = O.accept(tree.parent, tree.ids, pred, V)
        acc += n_path - 1
    mc = acc / n
    se = math.sqrt(expected * 4 / n) + 1e-3
    assert abs(mc - expected) < 4 * se, (mc, expected)


# ---------------------------------------------------------------- whole loop

def test_multistep_ppd_is_lossless(tiny):
    """Section 5.1 / Figure 5: with exact matching the generated text is that of
    the original model.  Trees carry the true greedy continuation along a random
    path (random depth) and random tokens elsewhere."""
    sh, W, m, kc0, vc0, L0, root = tiny
    kc, vc = O.copy_cache(kc0, vc0)
    steps, L, tok = 6, L0, root
    n_total = 0
    emitted = []
    rng = np.random.default_rng(7)
    for s in range(steps):
        tree = make_tree("candidates:10", sh.vocab, 3, 4, 500 + s, tok)
        truth = O.greedy_decode(m, kc, vc, L, tok, 6, "f32")
        node = int(rng.integers(tree.n_candidates))
        path_nodes = O.path_tokens(tree.parent, list(range(tree.T)), node)
        ids = tree.ids.copy()
        for k, nd in enumerate(path_nodes[1:]):
            ids[nd] = truth[k]
        res = O.verify_forward(m, kc, vc, L, ids, tree.parent, "f32")
        pred = O.argmax_first(res["logits"])
        path, n_path, nxt = O.accept(tree.parent, ids, pred, sh.vocab)
        assert n_path >= len(path_nodes)           # at least the planted path
        L = O.kv_compact(kc, vc, res["tree_k"], res["tree_v"], L, path)
        emitted += [int(ids[j]) for j in path[1:]] + [nxt]
        tok = nxt
        n_total += n_path
    ref = O.greedy_decode(m, kc0, vc0, L0, root, len(emitted), "f32")
    assert emitted == ref
    assert L == L0 + n_total


def test_kv_compact_commits_path_rows(tiny):
    sh, W, m, kc0, vc0, L, root = tiny
    tree = make_tree("candidates:10", sh.vocab, 3, 4, 31, root)
    res = O.verify_forward(m, kc0, vc0, L, tree.ids, tree.parent, "f32")
    depth, _ = O.build_mask(tree.parent)
    node = int(np.argmax(depth[:tree.n_candidates]))
    path = O.path_tokens(tree.parent, list(range(tree.T)), node)
    kc, vc = O.copy_cache(kc0, vc0)
    L2 = O.kv_compact(kc, vc, res["tree_k"], res["tree_v"], L, path)
    kr, vr = O.copy_cache(kc0, vc0)
    for j, nd in enumerate(path):
        O.decode_token(m, kr, vr, L + j, int(tree.ids[nd]), "f32")
    assert L2 == L + len(path)
    for l in range(sh.n_layers):
        assert np.abs(kc[l][:, :L2] - kr[l][:, :L2]).max() < 1e-12
        assert np.abs(vc[l][:, :L2] - vr[l][:, :L2]).max() < 1e-12


# ------------------------------------------------ next-step candidate generation

def _brute_rank(row, t):
    """Definition of a rank: the number of entries that beat entry t (a larger
    number, or an equal one at a smaller index; NaN beats nothing and loses to
    every number, NaNs among themselves by index)."""
    v = [float(x) for x in row]
    def beats(j, i):
        if math.isnan(v[i]):
            return (not math.isnan(v[j])) or j < i
        if math.isnan(v[j]):
            return False
        return v[j] > v[i] or (v[j] == v[i] and j < i)
    return sum(1 for j in range(len(v)) if j != t and beats(j, t))


def test_rank_order_matches_definition():
    rng = np.random.default_rng(11)
    for trial in range(40):
        n = int(rng.integers(1, 60))
        row = rng.integers(-3, 4, n).astype(np.float64)   # many ties
        if trial % 3 == 0:
            row[rng.integers(0, n, max(1, n // 5))] = np.nan
        order = O.rank_order(row)
        assert sorted(order.tolist()) == list(range(n))
        for r, t in enumerate(order):
            assert _brute_rank(row, int(t)) == r
        if not np.isnan(row).any():
            assert order[0] == O.argmax_first(row[None, :])[0]


def test_prompt_chain_handmade():
    V = 10
    # node 0 root; 1 candidate; 2,4,6 = root's chain (prompt ids 0, 1, 2);
    # 3,5,7 = candidate 1's chain; 8 = a stray prompt id 1 directly under 1
    parent = [-1, 0, 0, 1, 2, 3, 4, 5, 1]
    ids = [5, 7, V + 0, V + 0, V + 1, V + 1, V + 2, V + 2, V + 1]
    assert O.prompt_chain(parent, ids, V, 0) == [2, 4, 6]
    assert O.prompt_chain(parent, ids, V, 1) == [3, 5, 7]
    assert O.prompt_chain(parent, ids, V, 6) == []
    # a chain cut short: only prompt id 0 present
    assert O.prompt_chain([-1, 0, 1], [3, V, V + 5], V, 0) == [1]


def test_next_tree_ids_handmade():
    """Hand-computed: accepted node 1 with chain (3, 5); template root, ranks
    (0), (1), (0, 0), (0, 1) and one chain of 2 under the root."""
    V = 6
    parent = [-1, 0, 0, 1, 2, 3, 4]
    ids = [2, 4, V + 0, V + 0, V + 1, V + 1, 1]
    logits = np.zeros((7, V))
    logits[3] = [0.1, 0.9, 0.3, 0.9, -1.0, 0.2]   # depth-1 source: order 1, 3, 2, 5, 0, 4
    logits[5] = [2.0, 1.0, 3.0, 0.0, 3.0, -5.0]   # depth-2 source: order 2, 4, 0, 1, 3, 5
    tpl_parent = [-1, 0, 0, 1, 1, 0, 5]
    tpl_kind = [0, 0, 1, 0, 1, -1, -2]
    O.validate_template(tpl_parent, tpl_kind, 2)
    out = O.next_tree_ids(parent, ids, V, [0, 1], 4, logits, tpl_parent, tpl_kind)
    assert out.tolist() == [4, 1, 3, 2, 4, V + 0, V + 1]
    # accepted node without prompt tokens: every depth falls back to its own row
    logits[2] = [0, 0, 0, 0, 0, 9.0]
    out = O.next_tree_ids([-1, 0, 0], [2, 3, 5], V, [0, 2], 5, np.vstack([logits[:2], logits[2:3]]),
                          tpl_parent, tpl_kind)
    assert out.tolist() == [5, 5, 0, 5, 0, V + 0, V + 1]


@pytest.mark.parametrize("tpl_parent,tpl_kind", [
    ([-1, 0, 1], [0, -1, 0]),          # candidate under a prompt token
    ([-1, 0, 0], [0, 0, -2]),          # prompt id 1 directly under the root
    ([-1, 0, 1], [0, 0, -3]),          # prompt id 2 after a candidate
    ([-1, 0], [0, 16]),                # rank beyond the top-k limit
    ([-1, 0], [0, -4]),                # prompt id >= n_prompt
])
def test_validate_template_rejects(tpl_parent, tpl_kind):
    with pytest.raises(ValueError):
        O.validate_template(tpl_parent, tpl_kind, 3)


def test_closed_loop_with_generated_candidates_is_lossless(tiny):
    """Section 3's full guess-and-verify loop: each step's tree is the template
    filled from the previous step's outputs (bonus root, top-k of the accepted
    node's prompt tokens); the emitted tokens are the vanilla greedy sequence
    (Section 5.1: output identical to the original model)."""
    from synth.trees import make_template
    sh, W, m, kc0, vc0, L0, root = tiny
    tpl = make_template([(0,), (1,), (2,), (0, 0), (0, 1), (1, 0), (0, 0, 0)], 3)
    O.validate_template(tpl.parent, tpl.kind, sh.n_prompt)
    kc, vc = O.copy_cache(kc0, vc0)
    rng = np.random.default_rng(5)
    ids = rng.integers(0, sh.vocab, tpl.T)
    ids[0] = root
    ids[tpl.kind < 0] = sh.vocab + (-tpl.kind[tpl.kind < 0] - 1)
    L, emitted, accepted = L0, [], 0
    for s in range(6):
        res = O.verify_forward(m, kc, vc, L, ids, tpl.parent, "f32")
        pred = O.argmax_first(res["logits"])
        path, n_path, nxt = O.accept(tpl.parent, ids, pred, sh.vocab)
        L = O.kv_compact(kc, vc, res["tree_k"], res["tree_v"], L, path)
        emitted += [int(ids[j]) for j in path[1:]] + [nxt]
        accepted += n_path - 1
        ids = O.next_tree_ids(tpl.parent, ids, sh.vocab, path, nxt, res["logits"], tpl.parent,
                              tpl.kind)
        assert ids[0] == nxt
    ref = O.greedy_decode(m, kc0, vc0, L0, root, len(emitted), "f32")
    assert emitted == ref


# ------------------------------------------------- ensemble prompt tokens (EPT)

def test_ept_chains_realise_the_ensemble_mask():
    """The EPT appendix's ensemble mask: an EPT of group g sees the input
    tokens (here: the candidate path it hangs under) and the EPTs of group g
    at smaller or equal positions, nothing else.  The ancestor mask of a
    template with n_ept parallel chains per node is exactly that."""
    from synth.trees import make_template
    n_prompt, n_ept = 3, 3
    tpl = make_template([(0,), (1,), (0, 0)], n_prompt, n_ept)
    O.validate_template(tpl.parent, tpl.kind, n_prompt, n_ept)
    depth, anc = O.build_mask(tpl.parent)
    T = tpl.T
    # owner candidate, group and token distance of every EPT node, from the
    # template's kinds and the chain layout alone
    owner, group, dist = {}, {}, {}
    for i in range(1, T):
        k = int(tpl.kind[i])
        if k < 0:
            j, g = divmod(-k - 1, n_ept)
            group[i], dist[i] = g, j + 1
            o = i
            for _ in range(j + 1):
                o = int(tpl.parent[o])
            owner[i] = o

    def cand_path(c):
        out = {c}
        while c > 0:
            c = int(tpl.parent[c])
            out.add(c)
        return out

    for v in range(T):
        for u in range(T):
            if v in group:
                c = owner[v]
                want = (u in cand_path(c)) or (u in group and owner[u] == c and group[u] == group[v]
                                                and dist[u] <= dist[v])
            else:
                want = u in cand_path(v)
            assert bool(anc[v, u]) == want, (v, u)
        if v in group:
            assert depth[v] == depth[owner[v]] + dist[v]   # position = the token it stands for


def test_ept_mean_row_special_cases():
    rng = np.random.default_rng(21)
    x = rng.standard_normal(50).astype(np.float32)
    assert np.array_equal(O.ept_mean_row([x]), x)                      # one EPT: unchanged
    assert np.array_equal(O.ept_mean_row([x, x]), x)                   # (x + x) / 2 is exact
    a, b, c, d = (rng.integers(-1000, 1000, 50).astype(np.float32) for _ in range(4))
    exact = (a.astype(np.float64) + b + c + d) / 4.0                   # small integers: exact sums
    assert np.array_equal(O.ept_mean_row([a, b, c, d]).astype(np.float64), exact)
    assert np.array_equal(O.ept_mean_row([d, c, b, a]), O.ept_mean_row([a, b, c, d]))
    y = x.copy()
    y[7] = np.nan
    m = O.ept_mean_row([x, y])
    assert np.isnan(m[7]) and not np.isnan(np.delete(m, 7)).any()


def test_next_tree_ids_ept_handmade():
    """Two EPT groups; the averaged row ranks differently from either group's
    own row.  Accepted node 1 carries chains (3, 5) of group 0 and (4, 6) of
    group 1 (prompt ids 0, 2 and 1, 3); template: ranks (0), (1), (0, 0) and
    the two chains of length 2 under the root."""
    V, n_ept = 4, 2
    parent = [-1, 0, 0, 1, 1, 3, 4]
    ids = [2, 1, 3, V + 0, V + 1, V + 2, V + 3]
    logits = np.zeros((7, V), np.float32)
    logits[3] = [4.0, 0.0, 1.0, 2.0]     # group 0, distance 1: order 0, 3, 2, 1
    logits[4] = [-4.0, 2.0, 2.0, 0.0]    # group 1, distance 1: order 1, 2, 3, 0
    # mean [0, 1, 1.5, 1]: order 2, 1, 3, 0
    logits[5] = [1.0, 3.0, 0.0, 0.0]     # group 0, distance 2
    logits[6] = [1.0, -3.0, 0.0, 5.0]    # group 1, distance 2; mean [1, 0, 0, 2.5]: order 3, 0, 1, 2
    tpl_parent = [-1, 0, 0, 1, 0, 0, 4, 5]
    tpl_kind = [0, 0, 1, 0, -1, -2, -3, -4]
    O.validate_template(tpl_parent, tpl_kind, 2, n_ept)
    out = O.next_tree_ids(parent, ids, V, [0, 1], 3, logits, tpl_parent, tpl_kind, n_ept)
    assert out.tolist() == [3, 2, 1, 3, V + 0, V + 1, V + 2, V + 3]
    # identical groups: the mean is each group's row, as with one EPT
    logits[4], logits[6] = logits[3], logits[5]
    out = O.next_tree_ids(parent, ids, V, [0, 1], 3, logits, tpl_parent, tpl_kind, n_ept)
    one = O.next_tree_ids([-1, 0, 0, 1, 3], [2, 1, 3, V + 0, V + 1], V, [0, 1], 3,
                          logits[[0, 1, 2, 3, 5]], [-1, 0, 0, 1, 0, 4], [0, 0, 1, 0, -1, -2])
    assert out[:4].tolist() == one[:4].tolist()


@pytest.mark.parametrize("tpl_parent,tpl_kind", [
    ([-1, 0, 1], [0, -1, -4]),         # group 0 continued by group 1's distance-2 EPT
    ([-1, 0, 1], [0, -2, -3]),         # group 1 continued by group 0's distance-2 EPT
    ([-1, 0], [0, -7]),                # token distance 4 > 3
    ([-1, 0, 0], [0, 0, -3]),          # distance-2 EPT directly under the root
])
def test_validate_template_rejects_ept(tpl_parent, tpl_kind):
    O.validate_template([-1, 0, 1, 0, 3], [0, -1, -3, -2, -4], 3, 2)   # both groups, in order
    with pytest.raises(ValueError):
        O.validate_template(tpl_parent, tpl_kind, 3, 2)


def test_closed_loop_with_ept_candidates_is_lossless(tiny):
    """The guess-and-verify loop with two EPT groups per prompt token (each
    token distance has two embeddings, guesses from the averaged logits)
    still emits the vanilla greedy sequence."""
    import dataclasses
    from synth.trees import make_template
    sh, W, m, kc0, vc0, L0, root = tiny
    n_ept = 2
    sh2 = dataclasses.replace(sh, n_prompt=sh.n_prompt * n_ept)
    extra = np.random.default_rng(8).standard_normal((sh.n_prompt, sh.hidden)) * 0.02
    W2 = dict(W)
    W2["prompt_emb"] = np.vstack([O.to_f64(W["prompt_emb"]), extra])
    m2 = O.Model(sh2, W2)
    tpl = make_template([(0,), (1,), (2,), (0, 0), (0, 1), (1, 0), (0, 0, 0)], sh.n_prompt, n_ept)
    O.validate_template(tpl.parent, tpl.kind, sh.n_prompt, n_ept)
    kc, vc = O.copy_cache(kc0, vc0)
    rng = np.random.default_rng(6)
    ids = rng.integers(0, sh.vocab, tpl.T)
    ids[0] = root
    ids[tpl.kind < 0] = sh.vocab + (-tpl.kind[tpl.kind < 0] - 1)
    L, emitted = L0, []
    for s in range(5):
        res = O.verify_forward(m2, kc, vc, L, ids, tpl.parent, "f32")
        pred = O.argmax_first(res["logits"])
        path, n_path, nxt = O.accept(tpl.parent, ids, pred, sh.vocab)
        L = O.kv_compact(kc, vc, res["tree_k"], res["tree_v"], L, path)
        emitted += [int(ids[j]) for j in path[1:]] + [nxt]
        ids = O.next_tree_ids(tpl.parent, ids, sh.vocab, path, nxt,
                              res["logits"].astype(np.float32), tpl.parent, tpl.kind, n_ept)
    ref = O.greedy_decode(m, kc0, vc0, L0, root, len(emitted), "f32")
    assert emitted == ref


# ------------------------------------------------------------- tree sizing

def test_best_candidate_paths_is_optimal():
    """The rank paths of largest product maximise Proposition 1's sum over all
    candidate trees of that size (exhaustive search over prefix-closed sets of
    paths, depth <= 2, ranks < 3)."""
    import itertools
    rng = np.random.default_rng(41)
    for trial in range(6):
        p = rng.random((2, 3))
        paths = [(a,) for a in range(3)] + [(a, b) for a in range(3) for b in range(3)]
        val = {q: float(np.prod([p[j][r] for j, r in enumerate(q)])) for q in paths}
        for n in range(1, 6):
            best = 0.0
            for sub in itertools.combinations(paths, n):
                s = set(sub)
                if all(len(q) == 1 or q[:-1] in s for q in sub):
                    best = max(best, sum(val[q] for q in sub))
            got = O.best_candidate_paths(p, n)
            assert len(got) == n and all(len(q) == 1 or q[:-1] in set(got) for q in got)
            assert abs(sum(val[q] for q in got) - best) < 1e-12


def test_proposition1_on_sparse_template_monte_carlo():
    """Proposition 1 for a built template: draw the true token's rank at each
    distance independently from the table (or no match), verify with the
    oracle's exact-match acceptance, and average the accepted candidates."""
    from synth.trees import synthetic_accept_table
    p = synthetic_accept_table(3, 4)
    tp, tk, f = O.sparse_template(p, 9, 2)
    O.validate_template(tp, tk, 2)
    assert abs(O.prop1_expected_accepted(tp, tk, p) - f) < 1e-15
    K = p.shape[1]
    V = K + 1                      # token = rank; K = a token no candidate holds
    depth = O.template_depths(tp)
    ids = np.where(tk >= 0, tk, V + (-tk - 1))
    ids[0] = 0
    rng = np.random.default_rng(42)
    n, acc = 20000, 0
    for _ in range(n):
        r = [int(rng.choice(K + 1, p=np.append(p[d], 1 - p[d].sum()))) for d in range(3)]
        pred = np.array([r[int(depth[u])] if depth[u] < 3 else K for u in range(len(tp))])
        _, n_path, _ = O.accept(tp, ids, pred, V)
        acc += n_path - 1
    mc = acc / n
    se = math.sqrt(f * 3 / n) + 1e-3
    assert abs(mc - f) < 4 * se, (mc, f)


def test_sparse_template_layout():
    from synth.trees import synthetic_accept_table
    p = synthetic_accept_table()
    for n, n_prompt, n_ept in ((0, 3, 1), (15, 3, 1), (7, 3, 2), (20, 2, 1)):
        tp, tk, f = O.sparse_template(p, n, n_prompt, n_ept)
        O.validate_template(tp, tk, n_prompt, n_ept)
        assert len(tp) == 1 + n + (1 + n) * n_prompt * n_ept
        assert int(np.sum(tk[1:] >= 0)) == n
        assert O.template_depths(tp)[tk >= 0].max() <= p.shape[0]
    # more candidates never lower the expected accepted length
    fs = [O.sparse_template(p, n, 3)[2] for n in range(0, 32)]
    assert all(b >= a for a, b in zip(fs, fs[1:]))
