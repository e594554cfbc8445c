"""A captured step replays exactly: verify -> accept -> compact recorded once
as a HIP graph (torch.cuda.CUDAGraph) and replayed several times, with eager
work and synchronisations between the replays, gives every replay the eager
step's logits, greedy tokens, path and cache bit for bit.  The library
enqueues only kernels (no memset nodes), so nothing in the step depends on
being launched eagerly."""
import numpy as np
import pytest
import torch

import paper_2405_18628_amd as ppd
from gpu_cases import gpu_step, make_case, say, tree_for, tree_tensors, workspace
from synth import workload

pytestmark = pytest.mark.gpu


def test_graph_replay_equals_eager():
    case = make_case(workload("small"))
    tree = tree_for(case, spec="total:40")
    T, V, L = tree.T, case.shape.vocab, case.L
    say(f"[graph] small T={T} L={L}")
    ws = workspace(case, T)
    # plant the greedy continuation along the deepest candidate's root path
    # (a node's id = its parent's greedy token; changing a node leaves its
    # ancestors' logits alone), so the step accepts several nodes and the
    # compaction moves rows
    depth = ppd.ppd_build_tree_mask(tree.parent)[0]
    deep = max((i for i in range(T) if tree.ids[i] < V), key=lambda i: depth[i])
    chain = [deep]
    while chain[-1] != 0:
        chain.append(int(tree.parent[chain[-1]]))
    chain = chain[::-1]
    for node in chain[1:]:
        res = gpu_step(case, tree, ws, logits=False)
        tree.ids[node] = int(res["pred"][tree.parent[node]])
    tt = tree_tensors(tree)
    logits = torch.empty((T, V), device="cuda")
    pred = torch.empty(T, dtype=torch.int32, device="cuda")
    path = torch.empty(T, dtype=torch.int32, device="cuda")
    n_path = torch.empty(1, dtype=torch.int32, device="cuda")
    nxt = torch.empty(1, dtype=torch.int32, device="cuda")
    len_dev = torch.zeros(1, dtype=torch.int32, device="cuda")
    kv = ppd.KVCache(case.k, case.v, len_dev)
    k0, v0 = case.k.clone(), case.v.clone()

    def step():
        ppd.ppd_verify_step(case.model, kv, L, T, tt["ids"], tt["depth"], tt["mask"], ws, logits, pred)
        ppd.ppd_accept(T, tt["parent"], tt["ids"], pred, V, path, n_path, nxt, ws)
        ppd.ppd_kv_compact(case.model, kv, L, path, n_path)

    def outputs():
        n = int(n_path.item())
        return dict(logits=logits.clone(), pred=pred.clone(), path=path[:n].clone(), n=n,
                    nxt=int(nxt.item()), length=int(len_dev.item()), k=case.k.clone(), v=case.v.clone())

    def restore():
        case.k.copy_(k0)
        case.v.copy_(v0)
        logits.fill_(float("nan"))
        pred.fill_(-1)
        path.fill_(-7)
        n_path.zero_()
        nxt.zero_()
        len_dev.zero_()
        torch.cuda.synchronize()

    restore()
    step()
    torch.cuda.synchronize()
    ref = outputs()
    assert ref["length"] == L + ref["n"]
    assert ref["n"] == len(chain), (ref["n"], len(chain))

    # capture on a side stream after a warm-up there
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        restore()
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    restore()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    for r in range(4):
        restore()
        g.replay()
        torch.cuda.synchronize()
        got = outputs()
        say(f"[graph] replay {r}: n_path={got['n']}")
        assert torch.equal(got["logits"], ref["logits"]), f"replay {r}: logits"
        assert torch.equal(got["pred"], ref["pred"]), f"replay {r}: greedy tokens"
        assert got["n"] == ref["n"] and torch.equal(got["path"], ref["path"]), f"replay {r}: path"
        assert got["nxt"] == ref["nxt"] and got["length"] == ref["length"], f"replay {r}: bonus / length"
        assert torch.equal(got["k"], ref["k"]) and torch.equal(got["v"], ref["v"]), f"replay {r}: cache"
        # eager work between replays
        _ = (case.k.float().sum() + logits.nan_to_num().sum()).item()
    assert int(ppd.ppd_device_status(ws)) == 0
    restore()
