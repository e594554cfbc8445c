"""GPU parity of next-step candidate generation (ppd_next_tree) and the
device-only decode loop verify -> accept -> compact -> next tree.

The ids are integer selections: compared bit-exactly with the oracle's
`next_tree_ids` on the same float32 logits.  The closed loop on the fp32 tiny
decoder must emit exactly the vanilla greedy sequence (lossless)."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2405_18628_amd as ppd
from gpu_cases import check_logits, gpu_step, make_case, oracle_step, say, tree_tensors, workspace
from synth import workload
from synth.trees import RANK_PATHS_15, Tree, make_template, make_tree

pytestmark = pytest.mark.gpu


def _with_chains(tree: Tree, vocab: int, n_prompt: int, rng) -> Tree:
    """Add a prompt chain under every candidate that has none (so that any
    accepted node carries one), keeping topological order; some chains are
    cut short to exercise the fallback."""
    parent, ids = tree.parent.tolist(), tree.ids.tolist()
    has = set(parent[i] for i in range(len(parent)) if ids[i] == vocab)
    for c in range(tree.n_candidates):
        if c in has or len(parent) + n_prompt > 128:
            continue
        m = int(rng.integers(0, n_prompt + 1))
        prev = c
        for j in range(m):
            parent.append(prev)
            ids.append(vocab + j)
            prev = len(parent) - 1
    return Tree(np.asarray(parent, np.int32), np.asarray(ids, np.int32), tree.n_candidates)


def _synthetic_logits(T, V, rng, nan_rows=(), kind="ties"):
    if kind == "ties":
        x = rng.integers(-20, 21, (T, V)).astype(np.float32) * 0.25   # many ties
    elif kind == "normal":
        x = rng.standard_normal((T, V)).astype(np.float32)
    else:
        # "crowded": element i sits with 1023 others in a group i mod 1024;
        # groups whose number is below 15 mod 64 hold large values, those at
        # 15 mod 64 middling ones, so that thousands of elements beat every
        # 15th-best group maximum among 64 consecutive groups
        g = np.arange(V) % 1024 % 64
        x = rng.standard_normal((T, V)).astype(np.float32)
        x[:, g < 15] += 50.0
        x[:, g == 15] += 10.0
    for r in nan_rows:
        x[r, rng.integers(0, V, 7)] = np.nan
    return x


@pytest.mark.parametrize("V,spec,tpl_paths,seed,kind", [
    (1000, "candidates:10", RANK_PATHS_15, 1, "ties"),
    (32000, "total:40", RANK_PATHS_15, 2, "ties"),
    (37, "candidates:6", [(0,), (15,), (2,), (0, 3), (2, 0), (2, 0, 1)], 3, "ties"),
    (32000, "chain:1", [(0,), (1,), (0, 0)], 4, "ties"),
    (32000, "candidates:8", [(0,), (15,), (1,), (0, 15), (0, 3)], 5, "crowded"),
    (70001, "candidates:8", [(0,), (15,), (1,), (0, 15), (0, 3)], 6, "crowded"),
    (70001, "total:30", RANK_PATHS_15, 7, "normal"),
    (1023, "candidates:5", [(0,), (15,), (0, 7)], 8, "normal"),
    (40000, "total:30", RANK_PATHS_15, 9, "normal"),
    (65536, "candidates:8", [(0,), (15,), (1,), (0, 15), (0, 3)], 10, "crowded"),
])
def test_next_tree_ids_bit_exact(V, spec, tpl_paths, seed, kind):
    """Ranks from rows with many ties and NaNs, Gaussian rows, and rows
    crowded so that the candidate list overflows (then the ranks come from
    repeated maxima); rows longer than one register chunk (32768), rows read
    in float4 (vocab a multiple of 4) and element by element."""
    rng = np.random.default_rng(seed)
    n_prompt = 3
    if spec.startswith("chain"):
        tree = Tree(np.asarray([-1], np.int32), np.asarray([5], np.int32), 1)
    else:
        tree = make_tree(spec, V, n_prompt, 4, 100 + seed, 3)
    tree = _with_chains(tree, V, n_prompt, rng)
    tpl = make_template(tpl_paths, n_prompt)
    O.validate_template(tpl.parent, tpl.kind, n_prompt)
    T = tree.T
    tt = tree_tensors(tree)
    ws = torch.zeros(256, dtype=torch.uint8, device="cuda")
    for trial in range(6):
        a = int(rng.integers(0, tree.n_candidates))
        path = O.path_tokens(tree.parent, list(range(T)), a)
        logits = _synthetic_logits(T, V, rng, nan_rows=[trial % T] if trial % 2 else [], kind=kind)
        nxt = int(rng.integers(0, V))
        say(f"[next] V={V} T={T} tpl={tpl.T} accepted={a} trial={trial}")
        path_d = torch.tensor(path + [0] * (T - len(path)), dtype=torch.int32, device="cuda")
        n_path = torch.tensor([len(path)], dtype=torch.int32, device="cuda")
        nxt_d = torch.tensor([nxt], dtype=torch.int32, device="cuda")
        out = torch.full((tpl.T,), -9, dtype=torch.int32, device="cuda")
        ppd.ppd_next_tree(T, tt["parent"], tt["ids"], V, n_prompt, torch.from_numpy(logits).cuda(),
                          path_d, n_path, nxt_d, tpl.parent, tpl.kind, out, ws)
        torch.cuda.synchronize()
        ref = O.next_tree_ids(tree.parent, tree.ids, V, path, nxt, logits.astype(np.float64),
                              tpl.parent, tpl.kind)
        assert out.cpu().numpy().tolist() == ref.tolist()


def test_closed_loop_on_device_is_lossless():
    """Six decode steps with nothing but device calls between them (the
    template's parent, depth and mask are uploaded once): the emitted tokens
    equal the oracle's vanilla greedy continuation."""
    case = make_case(workload("tiny"))
    sh = case.shape
    tpl = make_template([(0,), (1,), (2,), (0, 0), (0, 1), (1, 0), (0, 0, 0)], 3)
    T = tpl.T
    depth, mask = ppd.ppd_build_tree_mask(tpl.parent)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    parent_d, depth_d, mask_d = dev(tpl.parent.astype(np.int32)), dev(depth), dev(mask.view(np.int64))
    rng = np.random.default_rng(5)
    ids0 = rng.integers(0, sh.vocab, T).astype(np.int32)
    ids0[0] = case.root
    ids0[tpl.kind < 0] = sh.vocab + (-tpl.kind[tpl.kind < 0] - 1)
    ids = dev(ids0)
    ws = workspace(case, T)
    logits = torch.empty((T, sh.vocab), dtype=torch.float32, device="cuda")
    pred = torch.empty(T, dtype=torch.int32, device="cuda")
    path = torch.zeros(T, dtype=torch.int32, device="cuda")
    n_path = torch.zeros(1, dtype=torch.int32, device="cuda")
    nxt = torch.zeros(1, dtype=torch.int32, device="cuda")
    nids = torch.zeros(T, dtype=torch.int32, device="cuda")
    len_dev = torch.zeros(1, dtype=torch.int32, device="cuda")
    kv = ppd.KVCache(case.k, case.v, len_dev)
    k0, v0 = case.k.clone(), case.v.clone()
    L, emitted = case.L, []
    for s in range(6):
        ppd.ppd_verify_step(case.model, kv, L, T, ids, depth_d, mask_d, ws, logits, pred)
        ppd.ppd_accept(T, parent_d, ids, pred, sh.vocab, path, n_path, nxt, ws)
        ppd.ppd_kv_compact(case.model, kv, L, path, n_path)
        ppd.ppd_next_tree(T, parent_d, ids, sh.vocab, sh.n_prompt, logits, path, n_path, nxt,
                          tpl.parent, tpl.kind, nids, ws)
        torch.cuda.synchronize()          # the test reads the tokens; the loop does not need to
        n = int(n_path.item())
        p = path[:n].cpu().tolist()
        cur = ids.cpu().tolist()
        emitted += [cur[j] for j in p[1:]] + [int(nxt.item())]
        say(f"[loop] step {s}: accepted {n - 1}, L={L}")
        L += n
        assert int(len_dev.item()) == L
        ids.copy_(nids)
    assert ppd.ppd_device_status(ws) == 0
    ref = O.greedy_decode(case.oracle_model, case.kc_host, case.vc_host, case.L, case.root,
                          len(emitted), "f32")
    assert emitted == ref
    case.k.copy_(k0)
    case.v.copy_(v0)


def _ept_tree(rank_paths, V, n_prompt, n_ept, rng, full=False) -> Tree:
    """A step's tree with ensemble prompt tokens: random candidate ids, and
    under the root and every candidate one chain per EPT group (group g:
    ids V + j * n_ept + g), each cut to a random length unless `full`."""
    parent, ids = [-1], [int(rng.integers(0, V))]
    node_of = {(): 0}
    for path in rank_paths:
        parent.append(node_of[tuple(path[:-1])])
        ids.append(int(rng.integers(0, V)))
        node_of[tuple(path)] = len(parent) - 1
    n_cand = len(parent)
    for c in range(n_cand):
        for g in range(n_ept):
            m = n_prompt if full else int(rng.integers(0, n_prompt + 1))
            prev = c
            for j in range(m):
                parent.append(prev)
                ids.append(V + j * n_ept + g)
                prev = len(parent) - 1
    assert len(parent) <= 128
    return Tree(np.asarray(parent, np.int32), np.asarray(ids, np.int32), n_cand)


@pytest.mark.parametrize("V,n_ept,kind,seed", [
    (32000, 2, "normal", 31),
    (1000, 3, "ties", 32),
    (37, 4, "ties", 33),
    (70001, 2, "crowded", 34),
    (40000, 2, "normal", 35),
    (32001, 3, "normal", 36),
])
def test_next_tree_ids_ept_bit_exact(V, n_ept, kind, seed):
    """Ensemble prompt tokens: the guesses rank the float32 mean of the EPT
    groups' rows; ids bit-exact against the oracle on the same float32
    logits, with chains of random length (some groups shorter, some absent)."""
    rng = np.random.default_rng(seed)
    n_prompt = 3
    paths = [(0,), (1,), (2,), (0, 0), (0, 1), (1, 0), (0, 0, 0)]
    tpl_paths = [(0,), (15,), (1,), (0, 3), (0, 0), (0, 0, 1)]
    tpl = make_template(tpl_paths, n_prompt, n_ept)
    O.validate_template(tpl.parent, tpl.kind, n_prompt, n_ept)
    ws = torch.zeros(256, dtype=torch.uint8, device="cuda")
    for trial in range(5):
        tree = _ept_tree(paths, V, n_prompt, n_ept, rng, full=trial == 0)
        T = tree.T
        tt = tree_tensors(tree)
        a = int(rng.integers(0, tree.n_candidates))
        path = O.path_tokens(tree.parent, list(range(T)), a)
        logits = _synthetic_logits(T, V, rng, nan_rows=[T - 1] if trial % 2 else [], kind=kind)
        nxt = int(rng.integers(0, V))
        say(f"[next-ept] V={V} n_ept={n_ept} T={T} tpl={tpl.T} accepted={a} trial={trial}")
        path_d = torch.tensor(path + [0] * (T - len(path)), dtype=torch.int32, device="cuda")
        n_path = torch.tensor([len(path)], dtype=torch.int32, device="cuda")
        nxt_d = torch.tensor([nxt], dtype=torch.int32, device="cuda")
        out = torch.full((tpl.T,), -9, dtype=torch.int32, device="cuda")
        ppd.ppd_next_tree(T, tt["parent"], tt["ids"], V, n_prompt, torch.from_numpy(logits).cuda(),
                          path_d, n_path, nxt_d, tpl.parent, tpl.kind, out, ws, n_ept=n_ept)
        torch.cuda.synchronize()
        ref = O.next_tree_ids(tree.parent, tree.ids, V, path, nxt, logits, tpl.parent, tpl.kind,
                              n_ept)
        assert out.cpu().numpy().tolist() == ref.tolist()


def test_closed_loop_with_ept_on_device_is_lossless():
    """The device-only decode loop with two EPT groups per prompt token (six
    prompt embeddings; guesses from the averaged logits) emits the oracle's
    vanilla greedy continuation."""
    import dataclasses
    case = make_case(workload("tiny"))
    sh = case.shape
    n_ept = 2
    sh2 = dataclasses.replace(sh, n_prompt=sh.n_prompt * n_ept)
    W2 = dict(case.W)
    gen = torch.Generator().manual_seed(9)
    extra = (torch.randn(sh.n_prompt, sh.hidden, generator=gen) * 0.02).to(
        W2["prompt_emb"].dtype).cuda()
    W2["prompt_emb"] = torch.cat([case.W["prompt_emb"], extra]).contiguous()
    model2 = ppd.Model(sh2, W2)
    tpl = make_template([(0,), (1,), (2,), (0, 0), (0, 1), (1, 0), (0, 0, 0)], sh.n_prompt, n_ept)
    T = tpl.T
    depth, mask = ppd.ppd_build_tree_mask(tpl.parent)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    parent_d, depth_d, mask_d = dev(tpl.parent.astype(np.int32)), dev(depth), dev(mask.view(np.int64))
    rng = np.random.default_rng(7)
    ids0 = rng.integers(0, sh.vocab, T).astype(np.int32)
    ids0[0] = case.root
    ids0[tpl.kind < 0] = sh.vocab + (-tpl.kind[tpl.kind < 0] - 1)
    ids = dev(ids0)
    ws = workspace(case, T)
    logits = torch.empty((T, sh.vocab), dtype=torch.float32, device="cuda")
    pred = torch.empty(T, dtype=torch.int32, device="cuda")
    path = torch.zeros(T, dtype=torch.int32, device="cuda")
    n_path = torch.zeros(1, dtype=torch.int32, device="cuda")
    nxt = torch.zeros(1, dtype=torch.int32, device="cuda")
    nids = torch.zeros(T, dtype=torch.int32, device="cuda")
    len_dev = torch.zeros(1, dtype=torch.int32, device="cuda")
    kv = ppd.KVCache(case.k, case.v, len_dev)
    k0, v0 = case.k.clone(), case.v.clone()
    L, emitted = case.L, []
    for s in range(5):
        ppd.ppd_verify_step(model2, kv, L, T, ids, depth_d, mask_d, ws, logits, pred)
        ppd.ppd_accept(T, parent_d, ids, pred, sh.vocab, path, n_path, nxt, ws)
        ppd.ppd_kv_compact(model2, kv, L, path, n_path)
        ppd.ppd_next_tree(T, parent_d, ids, sh.vocab, sh.n_prompt, logits, path, n_path, nxt,
                          tpl.parent, tpl.kind, nids, ws, n_ept=n_ept)
        torch.cuda.synchronize()
        n = int(n_path.item())
        p = path[:n].cpu().tolist()
        cur = ids.cpu().tolist()
        emitted += [cur[j] for j in p[1:]] + [int(nxt.item())]
        say(f"[loop-ept] step {s}: accepted {n - 1}, L={L}")
        L += n
        ids.copy_(nids)
    assert ppd.ppd_device_status(ws) == 0
    ref = O.greedy_decode(case.oracle_model, case.kc_host, case.vc_host, case.L, case.root,
                          len(emitted), "f32")
    assert emitted == ref
    case.k.copy_(k0)
    case.v.copy_(v0)


def test_verify_logits_on_ept_tree():
    """The verification forward on a tree with two EPT groups per prompt
    token (a candidate's chains side by side, six prompt embeddings): every
    node's logits, prompt nodes included, match the oracle at fp32 tolerance."""
    import dataclasses
    case = make_case(workload("tiny"))
    sh = case.shape
    n_ept = 2
    sh2 = dataclasses.replace(sh, n_prompt=sh.n_prompt * n_ept)
    W2 = dict(case.W)
    gen = torch.Generator().manual_seed(10)
    extra = (torch.randn(sh.n_prompt, sh.hidden, generator=gen) * 0.02).to(
        W2["prompt_emb"].dtype).cuda()
    W2["prompt_emb"] = torch.cat([case.W["prompt_emb"], extra]).contiguous()
    case2 = dataclasses.replace(case, shape=sh2, W=W2, model=ppd.Model(sh2, W2),
                                oracle_model=O.Model(sh2, W2))
    rng = np.random.default_rng(12)
    tree = _ept_tree([(0,), (1,), (2,), (0, 0), (0, 1), (1, 0), (0, 0, 0)], sh.vocab, sh.n_prompt,
                     n_ept, rng, full=True)
    ws = workspace(case2, tree.T)
    say(f"[ept-verify] T={tree.T}")
    gpu = gpu_step(case2, tree, ws)
    ref = oracle_step(case2, tree)
    check_logits(gpu["logits"], ref["logits"], sh.dtype)
