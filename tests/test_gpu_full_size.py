"""GPU parity at the benchmark workloads' full sizes.

Full width: the 1.4B, 7B, 13B (T in {16, 32, 64, 128}) and 7B-32k workloads
with their real hidden size, heads, FFN width, vocabulary, cache length and
tree, i.e. the same kernel launch configurations (tiles, K splits, attention
splits) that bench.py times -- those depend on the widths, T and L, not on
the number of layers -- with the decoder cut to one layer, every node
compared (and, where named, sampled nodes: a node's logits depend only on
its ancestors, so the oracle runs the ancestor closure of the sampled nodes
as its own tree).  The logits and greedy tokens of the full-depth steps are
compared with the oracle in test_gpu_full_depth.py.

Full depth, here: the 32-layer 7B benchmark configuration itself (and the
other workloads at full depth) checked by properties that hold at any size:
bitwise determinism, sampled nodes bitwise unchanged when every node outside
their ancestor chains gets other tokens, finite logits with a clean device
status, and acceptance / compaction bit-exact against the oracle's
acceptance on the GPU's greedy tokens.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2405_18628_amd as ppd
from gpu_cases import (check_logits, check_pred, gpu_step, make_case, say, subtree, tree_for,
                       workspace)
from synth import workload
from synth.trees import Tree

pytestmark = pytest.mark.gpu


def sample_nodes(tree, vocab, rng_seed=0):
    """Deepest candidate, node 1, the last node (end of a prompt chain), and
    one node drawn at random."""
    T = tree.T
    depth = np.zeros(T, dtype=np.int64)
    for i in range(1, T):
        depth[i] = depth[tree.parent[i]] + 1
    cand = [i for i in range(T) if tree.ids[i] < vocab]
    deepest = max(cand, key=lambda i: (depth[i], -i))
    rng = np.random.default_rng(rng_seed + T)
    nodes = {deepest, min(1, T - 1), T - 1, int(rng.integers(0, T))}
    return sorted(nodes)


def _compare_sampled(case, tree, res, nodes):
    sh = case.shape
    sub, keep = subtree(tree, nodes, sh.vocab)
    ref = O.verify_forward(case.oracle_model, case.kc_host, case.vc_host, case.L, sub.ids,
                           sub.parent, sh.dtype)
    at = [keep.index(n) for n in nodes]
    check_logits(res["logits"][nodes], ref["logits"][at], sh.dtype, "sampled logits")
    check_pred(res["pred"][nodes], ref["logits"][at], sh.dtype)
    L = case.L
    for l in range(sh.n_layers):
        gk = O.to_f64(case.k[l, :, [L + n for n in nodes], :])
        gv = O.to_f64(case.v[l, :, :, [L + n for n in nodes]]).transpose(0, 2, 1)
        check_logits(gk, ref["tree_k"][l][:, at, :], sh.dtype, f"tree K layer {l}")
        check_logits(gv, ref["tree_v"][l][:, at, :], sh.dtype, f"tree V layer {l}")


_CASES = {}


def _case(name, n_layers):
    key = (name, n_layers)
    if key not in _CASES:
        _CASES.clear()
        torch.cuda.empty_cache()
        _CASES[key] = make_case(workload(name, n_layers=n_layers), keep_layers=False)
    return _CASES[key]


@pytest.mark.parametrize("name,spec", [("1.4b", None), ("7b", None), ("7b", "root"),
                                       ("7b", "total:48"), ("7b", "total:112"),
                                       ("13b", "total:16"), ("13b", "total:32"),
                                       ("13b", "total:64"), ("13b", "total:96"),
                                       ("13b", "total:128"), ("7b-32k", None)])
def test_full_width_all_nodes(name, spec):
    """One decoder layer at the workload's full width: every node's logits,
    greedy token and tree keys / values against the oracle."""
    case = _case(name, 1)
    if spec == "root":
        tree = Tree(np.array([-1], np.int32), np.array([case.root], np.int32), 1)
    else:
        tree = tree_for(case, spec=spec)
    nodes = list(range(tree.T))
    say(f"[full-width] {name} T={tree.T} L={case.L} (all nodes)")
    ws = workspace(case, tree.T)
    res = gpu_step(case, tree, ws)
    assert ppd.ppd_device_status(ws) == 0
    _compare_sampled(case, tree, res, nodes)


def _accept_compact_bitexact(case, tree, res, ws):
    T, L = tree.T, case.L
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
    idx = torch.tensor(list(opath), device="cuda") + L
    k_rows = case.k[:, :, idx, :].clone()
    v_rows = case.v[:, :, :, idx].clone()
    ppd.ppd_kv_compact(case.model, ppd.KVCache(case.k, case.v), L, path, n_path)
    torch.cuda.synchronize()
    assert torch.equal(case.k[:, :, L:L + n, :], k_rows)
    assert torch.equal(case.v[:, :, :, L:L + n], v_rows)


@pytest.mark.parametrize("name", ["7b", "1.4b", "13b", "7b-32k"])
def test_full_depth_properties(name):
    case = _case(name, None)
    sh = case.shape
    tree = tree_for(case)
    say(f"[full-depth] {name} layers={sh.n_layers} T={tree.T} L={case.L}")
    ws = workspace(case, tree.T)
    a = gpu_step(case, tree, ws)
    b = gpu_step(case, tree, ws)
    assert np.isfinite(a["logits"]).all()
    assert ppd.ppd_device_status(ws) == 0
    assert np.array_equal(a["logits"], b["logits"]) and np.array_equal(a["pred"], b["pred"])
    # a node sees only its ancestors (Section 4.1): giving every node outside
    # the sampled nodes' ancestor closure other tokens (same T, L and launch
    # shapes) leaves the sampled nodes' logits bitwise unchanged -- masked
    # keys contribute exact zeros
    nodes = sample_nodes(tree, sh.vocab)
    _, keep = subtree(tree, nodes, sh.vocab)
    other = Tree(tree.parent.copy(), tree.ids.copy(), tree.n_candidates)
    rng = np.random.default_rng(7)
    changed = 0
    for i in range(tree.T):
        if i not in keep:
            if other.ids[i] < sh.vocab:
                other.ids[i] = (int(other.ids[i]) + 1 + int(rng.integers(0, sh.vocab - 1))) % sh.vocab
            else:
                other.ids[i] = sh.vocab + (int(other.ids[i]) - sh.vocab + 1) % sh.n_prompt
            changed += int(other.ids[i] != tree.ids[i])
    assert changed > 0
    c = gpu_step(case, other, ws)
    assert np.array_equal(c["logits"][nodes], a["logits"][nodes])
    assert np.array_equal(c["pred"][nodes], a["pred"][nodes])
    # the original tree's K/V rows back in place at L .. L + T - 1
    gpu_step(case, tree, ws)
    _accept_compact_bitexact(case, tree, a, ws)
