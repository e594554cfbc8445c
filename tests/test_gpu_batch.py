"""GPU parity of batched steps (ppd_verify_batch): several sequences, each
with its own cache, cached length and tree, share one pass over the weights.
The sequences are independent, so the reference for each is the oracle's
single-sequence step on it (there is no other arithmetic to check), and the
batched GPU rows must equal the GPU's own single-sequence step up to the
order of fp32 sums (the GEMMs' K split and tiling follow the step's total
token count, so a batch may add the same products in another order): logits
within 1e-3 + 1e-3 |x|, stored keys / values within one bf16 ulp (+ 1e-4),
greedy tokens equal wherever the single step's top-2 margin exceeds 2e-2.
Acceptance and compaction run per sequence on slices of the packed arrays,
bit-exact against the oracle."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2405_18628_amd as ppd
from gpu_cases import LazyCache, check_logits, check_pred, make_case, say, tree_tensors
from synth import workload
from synth.model import empty_kv, fill_kv_normal
from synth.trees import Tree, make_tree

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def small_case():
    return make_case(workload("small", cache_len=1500))


def _sequences(case, Ls, specs, seed):
    """Per sequence: its own cache (N(0,1) prefix of its own seed), L and tree."""
    sh = case.shape
    seqs = []
    for j, (L, spec) in enumerate(zip(Ls, specs)):
        cap = ((L + 128 + 63) // 64) * 64
        k, v = empty_kv(sh, cap, device="cuda")
        fill_kv_normal(k, v, L, seed + j)
        tree = make_tree(spec, sh.vocab, sh.n_prompt, 4, seed + 100 + j, 1 + j, 3)
        seqs.append(dict(L=L, tree=tree, k=k, v=v, kv=ppd.KVCache(k, v)))
    torch.cuda.synchronize()
    return seqs


def _packed(seqs):
    trees = [s["tree"] for s in seqs]
    parts = [tree_tensors(t) for t in trees]
    cat = {n: torch.cat([p[n] for p in parts]) for n in ("ids", "depth", "mask", "parent")}
    return trees, parts, cat


def _run_batch(case, seqs):
    trees, parts, cat = _packed(seqs)
    Ts = [t.T for t in trees]
    Tt = sum(Ts)
    ws = torch.empty(ppd.ppd_workspace_bytes(case.model, Tt, 4096), dtype=torch.uint8, device="cuda")
    ppd.ppd_workspace_init(ws)
    logits = torch.full((Tt, case.shape.vocab), float("nan"), device="cuda")
    pred = torch.full((Tt,), -1, dtype=torch.int32, device="cuda")
    ppd.ppd_verify_batch(case.model, [s["kv"] for s in seqs], [s["L"] for s in seqs], Ts,
                         cat["ids"], cat["depth"], cat["mask"], ws, logits, pred)
    torch.cuda.synchronize()
    return trees, parts, logits, pred, ws


def _same_step(lb, ls, pb, ps, kb, ks, vb, vs, what):
    """A sequence's rows of a batched step against its own single step."""
    a, b = lb.double().cpu().numpy(), ls.double().cpu().numpy()
    err = np.abs(a - b)
    # a stored key or value may round to the neighbouring bf16 value under
    # the other order of sums, which moves the logits by ~1e-4
    assert (err <= 1e-3 + 1e-3 * np.abs(b)).all(), f"{what}: logits differ by {err.max():.3e}"
    srt = np.sort(b, axis=1)
    decided = srt[:, -1] - srt[:, -2] > 2e-2
    assert np.array_equal(pb.cpu().numpy()[decided], ps.cpu().numpy()[decided]), what
    for x, y in ((kb, ks), (vb, vs)):
        # one bf16 ulp, plus the fp32 reordering noise of a K = 4096 sum
        # (~1e-5 of values of order 1) for keys near zero after RoPE
        xf, yf = x.float(), y.float()
        assert ((xf - yf).abs() <= 2 ** -7 * yf.abs() + 1e-4).all(), f"{what}: cache rows differ"


def _run_single(case, s):
    tt = tree_tensors(s["tree"])
    T = s["tree"].T
    ws = torch.empty(ppd.ppd_workspace_bytes(case.model, T, 4096), dtype=torch.uint8, device="cuda")
    ppd.ppd_workspace_init(ws)
    logits = torch.full((T, case.shape.vocab), float("nan"), device="cuda")
    pred = torch.full((T,), -1, dtype=torch.int32, device="cuda")
    ppd.ppd_verify_step(case.model, s["kv"], s["L"], T, tt["ids"], tt["depth"], tt["mask"], ws,
                        logits, pred)
    torch.cuda.synchronize()
    return logits, pred


@pytest.mark.parametrize("Ls,specs", [
    ([300, 1499, 37], ["total:40", "total:17", "candidates:10"]),
    ([0, 1, 700, 1024, 5, 64, 1200, 333], ["total:16"] * 8),
    ([1000], ["total:64"]),
    ([200, 900], ["total:64", "total:64"]),
    ([500, 0, 33], ["total:100", "total:8", "total:20"]),  # a sequence over 64 tokens: two tiles per wave
])
def test_batch_equals_single_sequences_and_oracle(small_case, Ls, specs):
    case = small_case
    sh = case.shape
    seqs = _sequences(case, Ls, specs, 7000 + Ls[0])
    say(f"[batch] B={len(seqs)} L={Ls} T={[s['tree'].T for s in seqs]}")
    trees, parts, logits, pred, ws = _run_batch(case, seqs)
    assert ppd.ppd_device_status(ws) == 0
    t0 = 0
    for j, s in enumerate(seqs):
        T = s["tree"].T
        lb, pb = logits[t0:t0 + T], pred[t0:t0 + T]
        # the tree's keys / values as the batched step stored them
        kb = s["k"][:, :, s["L"]:s["L"] + T].clone()
        vb = s["v"][:, :, :, s["L"]:s["L"] + T].clone()
        ls, ps = _run_single(case, s)
        _same_step(lb, ls, pb, ps, kb, s["k"][:, :, s["L"]:s["L"] + T], vb,
                   s["v"][:, :, :, s["L"]:s["L"] + T], f"sequence {j}")
        if j < 3:  # the oracle on a few sequences (it is the slow part)
            ref = O.verify_forward(case.oracle_model, LazyCache(s["k"], False, s["L"]),
                                   LazyCache(s["v"], True, s["L"]), s["L"], s["tree"].ids,
                                   s["tree"].parent, sh.dtype)
            check_logits(lb.cpu().numpy().astype(np.float64), ref["logits"], sh.dtype)
            check_pred(pb.cpu().numpy(), ref["logits"], sh.dtype)
        # acceptance and compaction of this sequence on its slices
        p = parts[j]
        path = torch.full((T,), -7, dtype=torch.int32, device="cuda")
        n_path = torch.zeros(1, dtype=torch.int32, device="cuda")
        nxt = torch.zeros(1, dtype=torch.int32, device="cuda")
        ppd.ppd_accept(T, p["parent"], p["ids"], pb.contiguous(), sh.vocab, path, n_path, nxt, ws)
        torch.cuda.synchronize()
        opath, on, onext = O.accept(s["tree"].parent, s["tree"].ids, pb.cpu().numpy(), sh.vocab)
        n = int(n_path.item())
        assert n == on and int(nxt.item()) == onext and path[:n].cpu().tolist() == list(opath)
        k_before, v_before = s["k"].clone(), s["v"].clone()
        ppd.ppd_kv_compact(case.model, s["kv"], s["L"], path, n_path)
        torch.cuda.synchronize()
        idx = torch.tensor(list(opath), device="cuda") + s["L"]
        assert torch.equal(s["k"][:, :, s["L"]:s["L"] + n], k_before[:, :, idx])
        assert torch.equal(s["v"][:, :, :, s["L"]:s["L"] + n], v_before[:, :, :, idx])
        t0 += T


def test_batch_full_width_7b_layer():
    """The 7B shape at full width (one decoder layer): four sequences of 16
    tree tokens with different cache lengths, in the benchmark's launch
    configuration; every sequence equals its own single-sequence step (up to
    the order of fp32 sums)."""
    case = make_case(workload("7b", n_layers=1), L=64)
    seqs = _sequences(case, [2048, 1024, 4000, 100], ["total:16"] * 4, 9100)
    say("[batch-7b] B=4 T=16 each")
    trees, parts, logits, pred, ws = _run_batch(case, seqs)
    t0 = 0
    for j, s in enumerate(seqs):
        T = s["tree"].T
        kb = s["k"][:, :, s["L"]:s["L"] + T].clone()
        vb = s["v"][:, :, :, s["L"]:s["L"] + T].clone()
        ls, ps = _run_single(case, s)
        _same_step(logits[t0:t0 + T], ls, pred[t0:t0 + T], ps, kb, s["k"][:, :, s["L"]:s["L"] + T],
                   vb, s["v"][:, :, :, s["L"]:s["L"] + T], f"sequence {j}")
        assert torch.isfinite(ls).all()
        t0 += T
