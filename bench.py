"""Benchmark of the PPD tree-verification step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload 7b] [--T 64] [--graph]
    python bench.py --sweep [--workload 13b]     # hardware-aware tree size
    python bench.py --batch-sweep                # several sequences per step
    python bench.py --stream-ceiling             # plain HBM read rates

A step is one pass of the whole hot path on one synthetic batch:
ppd_verify_step (forward over the T tree nodes, fp32 logits, greedy tokens)
-> ppd_accept -> ppd_kv_compact, enqueued on one stream.  The cache length L is
the same every step (the compaction writes past L, the next step overwrites).
Inputs are resident in HBM before timing starts.  Prints one JSON line.

--sweep measures the forward latency L_fp(T) of the sparse trees that
ppd_sparse_template builds for 0..31 candidates (3 prompt tokens under every
node: T = 4, 8, .., 128) and of vanilla decoding (T = 1), and prints one JSON
line per size and one with the size that maximises
Speedup = tau(T) / L_fp(T) against vanilla (Section 4.2), tau(T) = 1 + the
expected accepted candidates under the synthetic acceptance table.

--batch-sweep times batched steps (ppd_verify_batch over B sequences, each
with its own cache of L tokens and its own best sparse tree of T_s tokens,
then acceptance and compaction per sequence) for B = 1, 2, 4, 8 and T_s =
16, 32, next to vanilla batches (T_s = 1), and prints one JSON line each:
the speedup of PPD over vanilla decoding at the same batch size is
tau(T_s) x L(vanilla, B) / L(PPD, B).

The default line also times a planted-path step: the model's own greedy
continuation is planted along the deepest candidate chain of the same tree
(a node's id = its parent's greedy token), so acceptance takes that whole
chain and the compaction moves its rows inside the timed region; emitted
tokens per second there are the accepted tokens per step over its latency.
kernel_us are per-dispatch event times (each dispatch's own start to end,
start-up included), so they do not add up to the step.

--stream-ceiling reads 14.3 GB (the 7B step's algorithmic bytes) with the
library's read probe: as four launches over a 3.6 GB buffer, and as 80
launches over 179 MB slices (a gate/up weight), and prints the achieved
read rates next to the 8 TB/s peak.

The default workload is the Vicuna-7B-shaped decoder (32 layers, hidden 4096,
32 heads x 128, ffn 11008, vocab 32000, bf16, random weights) with a
2048-token KV prefix and a 64-node candidate tree (3 prompt tokens per leaf).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# the paper's mean tokens per step with PPD on MT-Bench (Table 1), by model
PAPER_TAU = {"1.4b": 2.43, "7b": 2.54, "13b": 2.44, "7b-32k": 2.54}
MFMA_BF16_PEAK_TFLOPS = 2500.0


def step_bytes(sh, L, T, n_path):
    """Algorithmic HBM bytes of one step: every weight matrix, norm gain and
    the LM head once, the KV prefix once, the tree K/V write, the T embedding
    rows, the fp32 logits write and the compaction's read + write."""
    H, F, nh, nkv, d, V, nl = (sh.hidden, sh.ffn, sh.n_heads, sh.n_kv_heads, sh.head_dim,
                               sh.vocab, sh.n_layers)
    es = 2 if sh.dtype == "bf16" else 4
    w = nl * (sh.qkv_rows * H + H * nh * d + 2 * F * H + H * F + 2 * H) + V * H + H
    kv_prefix = nl * nkv * L * d * 2
    tree_kv = nl * nkv * T * d * 2
    emb = T * H
    return (w + kv_prefix + tree_kv + emb) * es + T * V * 4 + 2 * n_path * nl * nkv * d * 2 * es


def step_flops(sh, L, T):
    per_tok = 2 * (sh.n_layers * (sh.qkv_rows * sh.hidden + sh.hidden * sh.n_heads * sh.head_dim
                                  + 3 * sh.ffn * sh.hidden) + sh.vocab * sh.hidden)
    attn = 4 * T * (L + T) * sh.n_heads * sh.head_dim * sh.n_layers
    return T * per_tok + attn


def gate_up_bytes(sh, T):
    """Algorithmic bytes of one gate/up launch: the [2F, H] weight, the
    [T, H] normalised operand and the [T, F] SwiGLU output."""
    return (2 * sh.ffn * sh.hidden + T * sh.hidden + T * sh.ffn) * 2


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="7b")
    ap.add_argument("--T", type=int, default=None)
    ap.add_argument("--L", type=int, default=None)
    ap.add_argument("--graph", action="store_true", help="replay the step as a HIP graph")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-layers", type=int, default=4,
                    help="decoder layers in the CPU oracle's timed sample")
    ap.add_argument("--sweep", action="store_true",
                    help="tree-size sweep: L_fp(T) of the best sparse trees and the speedup")
    ap.add_argument("--batch-sweep", action="store_true",
                    help="batched steps: B sequences per step, PPD against vanilla")
    ap.add_argument("--stream-ceiling", action="store_true",
                    help="plain HBM read rates (reductions over 14.3 GB)")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="only run a plain device copy of this many bytes (calibrates the "
                         "FETCH_SIZE / WRITE_SIZE counters) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (the step is a single-GPU kernel path); "
              f"--gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    if args.stream_ceiling:
        stream_ceiling()
        return
    if args.copy_bytes:
        n = args.copy_bytes // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n * 4, "launches": 3}), flush=True)
        return

    import paper_2405_18628_amd as ppd
    from synth import workload
    from synth.model import empty_kv, fill_kv_normal, make_weights
    from synth.trees import make_template, make_tree

    wl = workload(args.workload)
    sh = wl.shape
    L = wl.cache_len if args.L is None else args.L
    spec = wl.tree if args.T is None else f"total:{args.T}"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t0 = time.time()
    W = make_weights(sh, wl.seeds["weights"], device=dev)
    cap = ((L + 128 + 63) // 64) * 64
    k, v = empty_kv(sh, cap, device=dev)
    fill_kv_normal(k, v, L, wl.seeds["kv"])
    torch.cuda.synchronize()
    print(f"[bench] {wl.name}: inputs ready in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)

    tree = make_tree(spec, sh.vocab, sh.n_prompt, wl.max_depth, wl.seeds["tree"], 1, wl.max_fanout)
    T = tree.T
    depth, mask = ppd.ppd_build_tree_mask(tree.parent)
    todev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    ids_d, par_d, dep_d, mask_d = (todev(tree.ids), todev(tree.parent), todev(depth),
                                   todev(mask.view(np.int64)))
    model = ppd.Model(sh, W)
    kv = ppd.KVCache(k, v)
    if args.sweep:
        tree_size_sweep(args, ppd, wl, sh, model, kv, L, cap, dev)
        return
    if args.batch_sweep:
        del k, v, kv
        batch_sweep(args, ppd, wl, sh, model, L, cap, dev)
        return
    ws = torch.empty(ppd.ppd_workspace_bytes(model, T, cap), dtype=torch.uint8, device=dev)
    ppd.ppd_workspace_init(ws)
    logits = torch.empty((T, sh.vocab), device=dev)
    pred = torch.empty(T, dtype=torch.int32, device=dev)
    path = torch.empty(T, dtype=torch.int32, device=dev)
    n_path = torch.empty(1, dtype=torch.int32, device=dev)
    nxt = torch.empty(1, dtype=torch.int32, device=dev)

    def step():
        ppd.ppd_verify_step(model, kv, L, T, ids_d, dep_d, mask_d, ws, logits, pred)
        ppd.ppd_accept(T, par_d, ids_d, pred, sh.vocab, path, n_path, nxt, ws)
        ppd.ppd_kv_compact(model, kv, L, path, n_path)

    run = step
    if args.graph:
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            for _ in range(2):
                step()
        torch.cuda.current_stream().wait_stream(s)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        run = g.replay

    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    # one event between consecutive steps: the mean over the K steps and the
    # spread of the single steps
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    evs[0].record()
    for i in range(args.steps):
        run()
        evs[i + 1].record()
    torch.cuda.synchronize()
    ms = evs[0].elapsed_time(evs[-1]) / args.steps
    per_step_us = np.array([evs[i].elapsed_time(evs[i + 1]) * 1e3 for i in range(args.steps)])
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    n_acc = int(n_path.item())
    status = ppd.ppd_device_status(ws)

    # forward-only latency (verify without accept / compact)
    e0.record()
    for _ in range(args.steps):
        ppd.ppd_verify_step(model, kv, L, T, ids_d, dep_d, mask_d, ws, logits, pred)
    e1.record()
    torch.cuda.synchronize()
    fwd_ms = e0.elapsed_time(e1) / args.steps

    # per-kernel durations with HIP events on the step's stream (eager steps)
    kernels = {}
    for kind in ("qkv", "attention", "o_proj", "gate_up", "down", "lm_head"):
        n = 1 if kind == "lm_head" else sh.n_layers
        st = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        sp = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        keep = ppd.ppd_set_kernel_timer(kind, st, sp)
        tot, cnt = 0.0, 0
        for _ in range(args.steps):
            step()
            torch.cuda.synchronize()
            tot += sum(a.elapsed_time(b) for a, b in zip(st, sp))
            cnt += n
        ppd.ppd_set_kernel_timer(kind)
        del keep
        kernels[kind] = tot / cnt * 1e3  # us per launch

    # next-step candidate generation (ppd_next_tree) on this step's outputs,
    # with the 15-candidate template (1 + 15 candidates, 3 prompt tokens each)
    tpl = make_template()
    nids = torch.empty(tpl.T, dtype=torch.int32, device=dev)

    def next_tree():
        ppd.ppd_next_tree(T, par_d, ids_d, sh.vocab, sh.n_prompt, logits, path, n_path, nxt,
                          tpl.parent, tpl.kind, nids, ws)
    for _ in range(3):
        next_tree()
    torch.cuda.synchronize()
    next_us = 0.0
    st, sp = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    keep = ppd.ppd_set_kernel_timer("next_tree", [st], [sp])
    for _ in range(args.steps):
        next_tree()
        torch.cuda.synchronize()
        next_us += st.elapsed_time(sp) * 1e3 / args.steps
    ppd.ppd_set_kernel_timer("next_tree")
    del keep

    # the same with two EPT groups per prompt token (Section 3.2): the
    # 15-candidate template with two chains of 3 under every node (T = 112),
    # used as this step's tree, Gaussian logits, accepted path root -> node 1
    tpl2 = make_template(n_ept=2)
    gen = torch.Generator(device=dev)
    gen.manual_seed(wl.seeds["tokens"])
    logits2 = torch.randn((tpl2.T, sh.vocab), device=dev, generator=gen)
    ids2 = np.where(tpl2.kind < 0, sh.vocab + (-tpl2.kind - 1), 1 + np.arange(tpl2.T)).astype(np.int32)
    par2_d, ids2_d = todev(tpl2.parent.astype(np.int32)), todev(ids2)
    path2 = torch.zeros(tpl2.T, dtype=torch.int32, device=dev)
    path2[1] = 1
    n_path2 = torch.tensor([2], dtype=torch.int32, device=dev)
    nids2 = torch.empty(tpl2.T, dtype=torch.int32, device=dev)

    def next_tree_ept():
        ppd.ppd_next_tree(tpl2.T, par2_d, ids2_d, sh.vocab, sh.n_prompt, logits2, path2, n_path2,
                          nxt, tpl2.parent, tpl2.kind, nids2, ws, n_ept=2)
    for _ in range(3):
        next_tree_ept()
    torch.cuda.synchronize()
    next_ept_us = 0.0
    keep = ppd.ppd_set_kernel_timer("next_tree", [st], [sp])
    for _ in range(args.steps):
        next_tree_ept()
        torch.cuda.synchronize()
        next_ept_us += st.elapsed_time(sp) * 1e3 / args.steps
    ppd.ppd_set_kernel_timer("next_tree")
    del keep

    # planted path: the greedy continuation along the deepest candidate's
    # root path (changing a node leaves its ancestors' logits alone, so the
    # chain is planted top-down, one verify per node, untimed)
    depth_h = depth
    cand = [i for i in range(T) if tree.ids[i] < sh.vocab]
    deep = max(cand, key=lambda i: depth_h[i])
    chain = [deep]
    while chain[-1] != 0:
        chain.append(int(tree.parent[chain[-1]]))
    chain = chain[::-1]
    ids_p = tree.ids.copy()
    for node in chain[1:]:
        ppd.ppd_verify_step(model, kv, L, T, todev(ids_p), dep_d, mask_d, ws, logits, pred)
        ids_p[node] = int(pred[int(tree.parent[node])].item())
    ids_pd = todev(ids_p)

    def planted_step():
        ppd.ppd_verify_step(model, kv, L, T, ids_pd, dep_d, mask_d, ws, logits, pred)
        ppd.ppd_accept(T, par_d, ids_pd, pred, sh.vocab, path, n_path, nxt, ws)
        ppd.ppd_kv_compact(model, kv, L, path, n_path)
    for _ in range(args.warmup):
        planted_step()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        planted_step()
    e1.record()
    torch.cuda.synchronize()
    planted_ms = e0.elapsed_time(e1) / args.steps
    planted_n = int(n_path.item())

    alg = step_bytes(sh, L, T, n_acc)
    flops = step_flops(sh, L, T)
    gu_us = kernels["gate_up"]
    gu_bytes = gate_up_bytes(sh, T)
    achieved = gu_bytes / (gu_us * 1e-6) / 1e9
    # the headline metric names its configuration; other workloads say theirs
    if (args.workload, T, L) == ("7b", 64, 2048):
        metric = "verify-step latency (us) + achieved HBM GB/s, 7B shape, 64-token tree, 2k ctx"
    else:
        metric = (f"verify-step latency (us) + achieved HBM GB/s, {args.workload} shape, "
                  f"{T}-token tree, {L} ctx")
    out = {
        "metric": metric,
        "value": round(ms * 1e3, 1),
        "unit": "us",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": sh.dtype,
        "data": "synthetic (seeded random weights N(0,0.02), KV prefix N(0,1), random tree)",
        "config": {"workload": f"{sh.name} verify step", "layers": sh.n_layers,
                   "hidden": sh.hidden, "heads": sh.n_heads, "ffn": sh.ffn, "vocab": sh.vocab,
                   "tree_tokens": T, "cache_len": L, "graph": bool(args.graph)},
        "step_hbm_gbs": round(alg / (ms * 1e-3) / 1e9, 1),
        "step_roofline_frac": round(alg / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "step_alg_bytes": alg,
        "step_alg_tflops": round(flops / (ms * 1e-3) / 1e12, 2),
        "forward_us": round(fwd_ms * 1e3, 1),
        "step_us_p10_p50_p90": [round(float(np.percentile(per_step_us, q)), 1) for q in (10, 50, 90)],
        "tree_tokens_per_s": round(T / (ms * 1e-3), 1),
        "emitted_tokens_per_s": round(n_acc / (ms * 1e-3), 1),
        "planted_path": {"accepted_per_step": planted_n, "chain_nodes": len(chain),
                         "step_us": round(planted_ms * 1e3, 1),
                         "emitted_tokens_per_s": round(planted_n / (planted_ms * 1e-3), 1)},
        "kernel_us": {k2: round(v2, 2) for k2, v2 in kernels.items()},
        "kernel_us_note": "per-dispatch HIP events (start-up included; not additive)",
        "next_tree_us": round(next_us, 2),
        "next_tree_ept2_us": round(next_ept_us, 2),
        "device_status": status,
        "projected_tokens_per_s": (round(PAPER_TAU[args.workload] / (ms * 1e-3), 1)
                                   if args.workload in PAPER_TAU else None),
        "projection": ("the paper's mean accepted length on MT-Bench for this model "
                       f"(Table 1: {PAPER_TAU.get(args.workload)} tokens per step) over this "
                       "step's latency; a projection, not a measurement (random weights accept "
                       "little)"),
        "roofline": {"bound": "hbm", "kernel": "gate_up GEMM + SwiGLU",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": recorded_traffic(args.workload, T, L),
                     "alg_bytes_per_launch": gu_bytes, "avg_launch_us": round(gu_us, 2)},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(sh, W, k, v, L, tree, args.cpu_layers)
    print(json.dumps(out), flush=True)


def tree_size_sweep(args, ppd, wl, sh, model, kv, L, cap, dev):
    """Section 4.2's hardware-aware tree size on this GPU: L_fp(T) measured
    for the best sparse tree of each candidate count, tau(T) from
    Proposition 1 on the synthetic acceptance table, and the size with the
    largest tau(T) * L_fp(1) / L_fp(T)."""
    import numpy as np
    import torch
    from synth.trees import synthetic_accept_table

    p_table = synthetic_accept_table()
    rng = np.random.default_rng(wl.seeds["tree"])
    n_prompt = 3
    sizes = [(None, 1)] + [(n, 4 * (n + 1)) for n in range(0, 32)]
    ws = torch.empty(ppd.ppd_workspace_bytes(model, 128, cap), dtype=torch.uint8, device=dev)
    ppd.ppd_workspace_init(ws)
    logits = torch.empty((128, sh.vocab), device=dev)
    pred = torch.empty(128, dtype=torch.int32, device=dev)
    path = torch.empty(128, dtype=torch.int32, device=dev)
    n_path = torch.empty(1, dtype=torch.int32, device=dev)
    nxt = torch.empty(1, dtype=torch.int32, device=dev)
    todev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    rows, base = [], None
    for n_cand, T in sizes:
        if n_cand is None:                       # vanilla decoding: the root alone
            tp, tk, f = np.array([-1], np.int32), np.array([0], np.int32), 0.0
        else:
            tp, tk, f = ppd.ppd_sparse_template(p_table, n_cand, n_prompt)
        assert len(tp) == T
        ids = np.where(tk < 0, sh.vocab + (-tk - 1), rng.integers(0, sh.vocab, T)).astype(np.int32)
        depth, mask = ppd.ppd_build_tree_mask(tp)
        ids_d, par_d, dep_d, mask_d = todev(ids), todev(tp.astype(np.int32)), todev(depth), \
            todev(mask.view(np.int64))
        lg = logits[:T]

        def fwd():
            ppd.ppd_verify_step(model, kv, L, T, ids_d, dep_d, mask_d, ws, lg, pred)

        def step():
            fwd()
            ppd.ppd_accept(T, par_d, ids_d, pred, sh.vocab, path, n_path, nxt, ws)
            ppd.ppd_kv_compact(model, kv, L, path, n_path)

        res = {}
        for name, fn in (("forward", fwd), ("step", step)):
            for _ in range(args.warmup):
                fn()
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
            torch.cuda.synchronize()
            ev[0].record()
            for i in range(args.steps):
                fn()
                ev[i + 1].record()
            torch.cuda.synchronize()
            us = np.array([ev[i].elapsed_time(ev[i + 1]) * 1e3 for i in range(args.steps)])
            res[name] = (float(np.median(us)), float(np.percentile(us, 10)),
                         float(np.percentile(us, 90)))
        tau = 1.0 + f
        if base is None:
            base = res["forward"][0]
        row = {"sweep": sh.name, "cache_len": L, "tree_tokens": T,
               "candidates": 0 if n_cand is None else n_cand,
               "forward_us": [round(x, 1) for x in res["forward"]],
               "step_us": [round(x, 1) for x in res["step"]],
               "tau": round(tau, 4),
               "speedup_vs_vanilla": round(tau * base / res["forward"][0], 4),
               "step_hbm_gbs": round(step_bytes(sh, L, T, 1) / (res["step"][0] * 1e-6) / 1e9, 1)}
        rows.append(row)
        print(json.dumps(row), flush=True)
    best = max(rows, key=lambda r: r["speedup_vs_vanilla"])
    print(json.dumps({"sweep": sh.name, "cache_len": L, "best_tree_tokens": best["tree_tokens"],
                      "best_candidates": best["candidates"], "best_speedup": best["speedup_vs_vanilla"],
                      "tau": best["tau"], "note": "forward_us / step_us are [median, p10, p90] over "
                      f"{args.steps} steps; tau from the synthetic acceptance table"}), flush=True)


def batch_sweep(args, ppd, wl, sh, model, L, cap, dev):
    """Several sequences per step (ppd_verify_batch): step latency for B
    sequences with their own caches (L tokens each) and best sparse trees of
    T_s tokens, against vanilla decoding (T_s = 1) at the same B."""
    import numpy as np
    import torch
    from synth.model import empty_kv, fill_kv_normal
    from synth.trees import synthetic_accept_table

    p_table = synthetic_accept_table()
    todev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    B_max = 8
    caches = []
    for j in range(B_max):
        k, v = empty_kv(sh, cap, device=dev)
        fill_kv_normal(k, v, L, wl.seeds["kv"] + 100 * j)
        caches.append(ppd.KVCache(k, v))
    torch.cuda.synchronize()
    ws = torch.empty(ppd.ppd_workspace_bytes(model, 128, cap), dtype=torch.uint8, device=dev)
    ppd.ppd_workspace_init(ws)
    logits = torch.empty((128, sh.vocab), device=dev)
    pred = torch.empty(128, dtype=torch.int32, device=dev)
    path = torch.empty(128, dtype=torch.int32, device=dev)
    n_path = torch.empty(B_max, dtype=torch.int32, device=dev)
    nxt = torch.empty(B_max, dtype=torch.int32, device=dev)
    rng = np.random.default_rng(wl.seeds["tree"])
    base = {}
    for Ts in (1, 16, 32):
        if Ts == 1:
            tp, tk, f = np.array([-1], np.int32), np.array([0], np.int32), 0.0
        else:
            tp, tk, f = ppd.ppd_sparse_template(p_table, Ts // 4 - 1, 3)
        depth, mask = ppd.ppd_build_tree_mask(tp)
        for B in (1, 2, 4, 8):
            if B * Ts > 128:
                continue
            ids = [np.where(tk < 0, sh.vocab + (-tk - 1), rng.integers(0, sh.vocab, Ts))
                   for _ in range(B)]
            ids_d = todev(np.concatenate(ids).astype(np.int32))
            dep_d = todev(np.tile(depth, B))
            mask_d = todev(np.tile(mask.view(np.int64), (B, 1)))
            par_d = todev(np.tile(tp.astype(np.int32), B))
            kvs, Ls = caches[:B], [L] * B

            def step():
                ppd.ppd_verify_batch(model, kvs, Ls, [Ts] * B, ids_d, dep_d, mask_d, ws,
                                     logits[:B * Ts], pred[:B * Ts])
                for j in range(B):
                    o = j * Ts
                    ppd.ppd_accept(Ts, par_d[o:o + Ts], ids_d[o:o + Ts], pred[o:o + Ts], sh.vocab,
                                   path[o:o + Ts], n_path[j:j + 1], nxt[j:j + 1], ws)
                    ppd.ppd_kv_compact(model, kvs[j], L, path[o:o + Ts], n_path[j:j + 1])

            for _ in range(args.warmup):
                step()
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
            torch.cuda.synchronize()
            ev[0].record()
            for i in range(args.steps):
                step()
                ev[i + 1].record()
            torch.cuda.synchronize()
            us = np.array([ev[i].elapsed_time(ev[i + 1]) * 1e3 for i in range(args.steps)])
            med = float(np.median(us))
            tau = 1.0 + f
            if Ts == 1:
                base[B] = med
            row = {"batch_sweep": sh.name, "cache_len": L, "sequences": B, "tree_tokens_each": Ts,
                   "step_us": [round(med, 1), round(float(np.percentile(us, 10)), 1),
                               round(float(np.percentile(us, 90)), 1)],
                   "tau": round(tau, 4),
                   "tree_tokens_per_s": round(B * Ts / (med * 1e-6), 1),
                   "projected_tokens_per_s": round(B * tau / (med * 1e-6), 1),
                   "speedup_vs_vanilla_same_batch": round(tau * base[B] / med, 4)}
            print(json.dumps(row), flush=True)


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gate_up_gemm_7b_hbm_traffic.md")
GEMM_SOURCE = os.path.join(ROOT, "paper_2405_18628_amd", "csrc", "k_gemm.hip")


def recorded_traffic(workload_name, T, L):
    """HBM bytes per gate/up launch measured with the FETCH_SIZE and
    WRITE_SIZE counters (calibrated against a plain copy), as recorded in the
    profile summary; None unless that summary was taken on this workload and
    on the GEMM source as it is now (its SHA-256 is recorded with it)."""
    import hashlib
    import re
    try:
        txt = open(TRAFFIC_FILE).read()
    except OSError:
        return None
    fields = dict(re.findall(r"^- (\w+): (\S+)\s*$", txt, re.M))
    src_sha = hashlib.sha256(open(GEMM_SOURCE, "rb").read()).hexdigest()
    if (fields.get("source_sha256") != src_sha or fields.get("workload") != workload_name
            or fields.get("tree_tokens") != str(T) or fields.get("cache_len") != str(L)):
        return None
    try:
        return int(float(fields["hbm_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def cpu_baseline(sh, W, k, v, L, tree, n_sample):
    """The oracle (float64 numpy, BLAS threads = host cores) on the same step:
    the full-depth forward + acceptance over the same tree and cache, median
    of 3 runs (the weights and caches are copied from the device and
    converted to float64 before timing; n_sample is unused: the whole step
    is the sample).  Beside it, single-thread latencies of the oracle on the
    tiny fp32 decoder and the MobileLLaMA-1.4B shape (configurations 0 and 1
    with their own trees and caches), one run each after a warm-up run for
    the tiny one."""
    import numpy as np
    import oracle as O
    from threadpoolctl import threadpool_info, threadpool_limits
    cores = max((i.get("num_threads", 1) for i in threadpool_info()), default=os.cpu_count())

    def timed(shape, Wd, kd, vd, Ld, tr, runs):
        m = O.Model(shape, Wd, keep_layers=True)
        for l in range(shape.n_layers):
            m.layer(l)
            if l % 8 == 7:
                print(f"[bench] oracle {shape.name}: {l + 1} layers converted", file=sys.stderr, flush=True)
        _ = m.lm_head
        kc = [O.to_f64(kd[l, :, :Ld, :]) for l in range(shape.n_layers)]
        vc = [O.to_f64(vd[l, :, :, :Ld]).transpose(0, 2, 1) for l in range(shape.n_layers)]
        out = []
        for _ in range(runs):
            t0 = time.perf_counter()
            res = O.verify_forward(m, kc, vc, Ld, tr.ids, tr.parent, shape.dtype)
            pred = O.argmax_first(res["logits"])
            O.accept(tr.parent, tr.ids, pred, shape.vocab)
            out.append(time.perf_counter() - t0)
            print(f"[bench] oracle {shape.name}: run {len(out)} {out[-1]:.2f} s", file=sys.stderr, flush=True)
        del m, kc, vc
        return out

    full = timed(sh, W, k, v, L, tree, 3)
    single = {}
    with threadpool_limits(1):
        from synth import workload
        from synth.model import empty_kv, fill_kv_normal, make_weights
        from synth.trees import make_tree
        for name in ("tiny", "1.4b"):
            wl = workload(name)
            shp = wl.shape
            Wt = make_weights(shp, wl.seeds["weights"], device="cpu")
            kt, vt = empty_kv(shp, wl.cache_len + 64, device="cpu")
            fill_kv_normal(kt, vt, wl.cache_len, wl.seeds["kv"])
            tr = make_tree(wl.tree, shp.vocab, shp.n_prompt, wl.max_depth, wl.seeds["tree"], 1,
                           wl.max_fanout)
            r = timed(shp, Wt, kt, vt, wl.cache_len, tr, 2 if name == "tiny" else 1)
            single[shp.name] = {"us": round(r[-1] * 1e6, 1), "tree_tokens": tr.T,
                                "cache_len": wl.cache_len, "layers": shp.n_layers}
            del Wt, kt, vt
    return {"value": round(float(np.median(full)) * 1e6, 1), "unit": "us", "cores": int(cores),
            "kind": "oracle",
            "sample": (f"the whole step: oracle forward over all {sh.n_layers} decoder layers + "
                       f"acceptance, the same {tree.T}-node tree and {L}-token cache, median of 3 "
                       f"runs ({', '.join(f'{t:.2f}' for t in full)} s)"),
            "single_thread_us": single}


def stream_ceiling():
    """Plain read rates of HBM with the library's read probe (one workgroup
    per compute unit streaming its contiguous piece with 16-byte
    non-temporal loads): 14.3 GB read as four launches over one 3.6 GB
    buffer, and as 80 launches over 179 MB slices of it (the size of a
    gate/up weight, launched back to back like the step's kernels); each
    timed with events around the launches, median of repeats."""
    import numpy as np
    import torch
    import paper_2405_18628_amd as ppd
    n = 900 * (1 << 20)  # floats: 3.77 GB
    buf = torch.ones(n, dtype=torch.float32, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    sl = 179 * (1 << 20) // 4
    nsl = n // sl

    def rate(fn, nbytes, reps):
        ts = []
        for _ in range(reps + 1):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b) * 1e-3)
        return nbytes / float(np.median(ts[1:])) / 1e9

    def big():
        for _ in range(4):
            ppd.ppd_read_probe(buf, sink)

    def chain():
        for i in range(80):
            ppd.ppd_read_probe(buf[(i % nsl) * sl:(i % nsl + 1) * sl], sink)
    r_big = rate(big, 4 * n * 4, 3)
    r_chain = rate(chain, 80 * sl * 4, 3)
    print(json.dumps({"stream_ceiling": {"big_launch_gbs": round(r_big, 1), "big_launch_bytes": n * 4,
                                         "chain_80x179MB_gbs": round(r_chain, 1),
                                         "chain_launch_bytes": sl * 4, "peak_gbs": HBM_PEAK_GBS,
                                         "big_frac": round(r_big / HBM_PEAK_GBS, 4),
                                         "chain_frac": round(r_chain / HBM_PEAK_GBS, 4),
                                         "method": "ppd_read_probe launches, HIP events"}}),
          flush=True)

if __name__ == "__main__":
    main()
