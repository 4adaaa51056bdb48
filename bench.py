#!/usr/bin/env python3
"""CompKV decode-step benchmark on one MI355X.

A step is one decode step of one attention layer: append the new token (cache row + active-block
summary), score and select blocks, then the compensated sparse attention. The timed step is the fused
call compkv_decode_step; the same step as three separate calls (compkv_append_stats,
compkv_score_select, compkv_sparse_decode) is timed beside it. Steps rotate over `--layers` resident
layer copies so the working set exceeds the 256 MB Infinity Cache and every step reads HBM, as
consecutive layers of a model do. The dense baseline step writes the same cache row and runs
compkv_dense_decode.

Prints one JSON line. `value` is microseconds per decode step per layer (lower is better); the line
also carries the achieved HBM bandwidth of the step and of its dominant kernel against the MI355X peak
(8 TB/s), the speedup over the dense decode, and the CPU oracle's time for the same step.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

HBM_PEAK_GBPS = 8000.0
PATH_NAMES = {1: "chunked", 2: "one_group", 3: "chunked_exact", 4: "stream"}
# extra budgets timed beside a workload's own (the long-context layer's budget sweep)
BUDGET_SWEEPS = {"long_128k": (32, 64, 128)}


def step_kernels(path: int) -> str:
    """The dispatches of one compkv_decode_step call on the given launch shape."""
    return {1: "compkv_decode_step: chunk scoring (append, compensation stream), selection, exact items, merge",
            2: "compkv_decode_step: one-group scoring and selection (append), exact and compensation items, merge",
            3: "compkv_decode_step: chunk scoring (append), then one launch of selection, compensation stream, "
               "exact items and merge",
            4: "compkv_decode_step: group scoring (append), then one launch of selector, compensation stream, "
               "exact items and merge",
            }[path]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=400)
    ap.add_argument("--warmup", type=int, default=40)
    ap.add_argument("--workload", default="long_128k")
    ap.add_argument("--budget", type=int, default=None, help="override the workload's block budget")
    ap.add_argument("--context", type=int, default=0,
                    help="override the workload's tokens per sequence (a context sweep of one layer shape)")
    ap.add_argument("--layers", type=int, default=0, help="resident layer copies (0: enough for > 1 GB)")
    ap.add_argument("--select-path", choices=["auto", "chunked", "one_group", "chunked_exact", "stream"],
                    default="auto",
                    help="scoring / selection launch shape (auto: one workgroup per unit where it fits)")
    ap.add_argument("--score-kind", choices=["compkv", "mass", "first_order"], default="compkv",
                    help="block score: the CompKV score or an ablation variant (mass only, first-order mass)")
    ap.add_argument("--compensation", choices=["mean", "drop"], default="mean",
                    help="decode of the omitted blocks: Mean compensation or Drop")
    ap.add_argument("--n-var-groups", type=int, default=0, help="override r, the variance groups per block")
    ap.add_argument("--host-kv", action="store_true",
                    help="offload tier: K/V caches in pinned host memory, read across the host link")
    ap.add_argument("--host-summaries", action="store_true",
                    help="with --host-kv: the fp32 summaries in pinned host memory too (the paper's layout)")
    ap.add_argument("--page-tokens", type=int, default=0,
                    help="paged K/V cache with pages of this many tokens, randomly permuted (0: contiguous)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=8.0,
                    help="oracle time budget of each CPU-baseline leg (one thread, then all host threads)")
    ap.add_argument("--no-sweep", action="store_true", help="skip the extra budgets of the workload's sweep")
    ap.add_argument("--only", choices=["all", "sparse", "dense", "fused"], default="all",
                    help="limit the timed work (for profiler runs): sparse = fused step and separate calls, "
                         "fused = the fused step alone")
    ap.add_argument("--eager", action="store_true",
                    help="launch kernels directly instead of replaying HIP graphs (for counter collection)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run three device copies of MIB MiB (reference reading for HBM byte counters)")
    return ap.parse_args()


def algorithmic_bytes(w, budget, sel_counts, compensate=True):
    """Bytes the method must move per step (all units), split by kernel.

    score_select: mean key (4d) and grouped variances (4r) of every block, the queries (2Gd bytes of
    bf16), and the selected ids written (4K).
    sparse_decode: bf16 keys and values of the selected tokens (4d per token), the fp32 mean value of
    every omitted block (4d; none for the Drop decode), the queries and the fp32 output (4Gd).
    append_stats: the new key/value (4d), the cache row written (4d), the active block's summary read
    and written (2 (8d + 4r)).
    """
    d, r, G, B, n = w.head_dim, w.n_var_groups, w.group, w.block_size, w.context
    X = -(-n // B)
    units = w.units
    last_len = n - (X - 1) * B
    score = units * (X * (4 * d + 4 * r) + 2 * G * d + 4 * budget)
    dec = 0
    for sel in sel_counts:  # per unit: list of selected ids
        tokens = sum(last_len if b == X - 1 else B for b in sel)
        dec += tokens * 4 * d + (X - len(sel)) * 4 * d * compensate + 2 * G * d + 4 * G * d
    app = units * (8 * d + 2 * (8 * d + 4 * r))
    dense = units * (n * 4 * d + 2 * G * d + 4 * G * d)
    return dict(score_select=score, sparse_decode=dec, append_stats=app, dense_decode=dense)


def measured_traffic(workload: str, call: str):
    """HBM bytes per call from the committed rocprofv3 byte counters (profiles/hbm_traffic.json), or None
    when the kernel sources changed since the counters were taken."""
    import glob
    import hashlib

    here = os.path.dirname(os.path.abspath(__file__))
    try:
        rec = json.load(open(os.path.join(here, "profiles", "hbm_traffic.json")))
    except (OSError, ValueError):
        return None
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(here, "paper_2609_26300_amd", "csrc", "*"))):
        h.update(open(f, "rb").read())
    if rec.get("source_sha256") != h.hexdigest():
        return None
    return rec.get("traffic_bytes", {}).get(workload, {}).get(call)


def host_cpu():
    """(model name, logical CPUs visible, threads the all-core oracle run may use) of this host."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    visible = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    # at most 16 threads: the CPU share of one GPU on a shared box, whatever the machine shows
    return model, os.cpu_count() or 1, max(1, min(16, visible))


def cpu_baseline(w, budget, Kb, Vb, qb, seconds):
    """The oracle (plain C, fp64) on the same step: score, select, compensated decode of every unit,
    from prebuilt fp64 summaries. Timed once on one thread and once on all host threads (one unit per
    thread at a time; the C calls release the interpreter lock)."""
    from concurrent.futures import ThreadPoolExecutor

    import oracle

    scale = 1.0 / math.sqrt(w.head_dim)
    B, r, G, n = w.block_size, w.n_var_groups, w.group, w.context
    units = [(b, h) for b in range(w.batch) for h in range(w.n_kv_heads)]
    model, nproc, threads = host_cpu()
    with ThreadPoolExecutor(max_workers=threads) as ex:
        built = list(ex.map(lambda u: oracle.block_stats(Kb[u[0], u[1]], Vb[u[0], u[1]], n, B, r), units))
    stats = dict(zip(units, built))

    def unit(u):
        b, h = u
        km, dv, vm = stats[b, h]
        q = qb[b, h * G:(h + 1) * G]
        sc = oracle.block_scores(q, km, dv, n, B, r, scale)
        sel = oracle.select(sc["score"], budget)
        oracle.sparse_decode(q, Kb[b, h], Vb[b, h], km, vm, n, B, scale, sel)

    def timed(nthreads):
        reps, t0 = 0, time.perf_counter()
        with ThreadPoolExecutor(max_workers=nthreads) as ex:
            while True:
                if nthreads == 1:
                    for u in units:
                        unit(u)
                else:
                    list(ex.map(unit, units))
                reps += 1
                el = time.perf_counter() - t0
                if el >= seconds:
                    return el / reps * 1e6, reps

    one_us, one_reps = timed(1)
    all_us, all_reps = timed(threads)
    return dict(value=round(all_us, 1), unit="us/decode-step/layer", cores=threads, kind="oracle",
                sample=f"{all_reps} full decode steps of the {w.name} layer ({len(units)} units) on {threads} "
                       f"threads, and {one_reps} on one thread: block scores, selection and compensated decode "
                       f"from prebuilt fp64 summaries",
                one_core_value=round(one_us, 1), host_cpu=model, nproc=nproc)


def run_streaming(args, w):
    """The streaming workload: every layer's cache is prefilled with `w.context` tokens, then
    `w.decode_steps` decode steps each append one token per sequence and run the whole step (fresh
    queries per step) on every layer. Each step is one captured graph (its layers in order); a first
    pass over all steps warms up (an append at position n rewrites the same row and recomputes the
    same active-block summary, so the timed second pass repeats exactly the same work). Reports the
    mean per step and layer over all steps and over steps 193-208."""
    import torch

    import paper_2609_26300_amd as P
    from workloads import gen_layer, gen_queries

    budget = args.budget or w.budget_blocks
    n0, T, Lyr = w.context, w.decode_steps, w.layers
    dev = "cuda"
    scale = 1.0 / math.sqrt(w.head_dim)
    dims = P.make_dims(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.block_size, w.n_var_groups,
                       w.capacity, max_seq_len=w.capacity)

    def to_dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(dev)

    Ks, Vs, Kn, Vn, summ, Q = [], [], [], [], [], []
    prefill = torch.full((w.batch,), n0, dtype=torch.int32, device=dev)
    host0 = None
    for L in range(Lyr):
        Kb, Vb, _ = gen_layer(w, L)
        if L == 0:
            host0 = (Kb, Vb)
        K, V = to_dev(Kb), to_dev(Vb)
        # the appended tokens, one [batch][Hkv][d] row per step; the cache holds only the prefill
        Kn.append(K[:, :, n0:n0 + T].permute(2, 0, 1, 3).contiguous())
        Vn.append(V[:, :, n0:n0 + T].permute(2, 0, 1, 3).contiguous())
        K[:, :, n0:] = 0
        V[:, :, n0:] = 0
        s = P.alloc_summaries(dims)
        P.compkv_build_stats(dims, K, V, prefill, s.kmean, s.dvar, s.vmean)
        Ks.append(K)
        Vs.append(V)
        summ.append(s)
        Q.append(to_dev(np.stack([np.stack([gen_queries(w, L, b, t) for b in range(w.batch)]) for t in range(T)])))
    seq_before = [torch.full((w.batch,), n0 + t, dtype=torch.int32, device=dev) for t in range(T)]
    seq_after = [torch.full((w.batch,), n0 + t + 1, dtype=torch.int32, device=dev) for t in range(T)]
    units = (w.batch, w.n_kv_heads)
    ws = P.alloc_workspace(dims, budget)
    sel = torch.empty((*units, budget), dtype=torch.int32, device=dev)
    n_sel = torch.empty(units, dtype=torch.int32, device=dev)
    blk_logit = torch.empty((*units, w.group, dims.xcap), dtype=torch.float32, device=dev)
    out = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=torch.float32, device=dev)
    lse = torch.empty((w.batch, w.n_q_heads), dtype=torch.float32, device=dev)
    params = P.CompkvSelectParams(budget, 1, 2, scale)
    torch.cuda.synchronize()

    def fused(L, t):
        s = summ[L]
        P.compkv_decode_step(dims, params, Q[L][t], Ks[L], Vs[L], Kn[L][t], Vn[L][t], seq_after[t], s.kmean,
                             s.dvar, s.vmean, sel, n_sel, blk_logit, None, out, lse, ws)

    def separate(L, t):
        s = summ[L]
        P.compkv_append_stats(dims, Ks[L], Vs[L], Kn[L][t], Vn[L][t], seq_before[t], s.kmean, s.dvar, s.vmean)
        P.compkv_score_select(dims, params, Q[L][t], s.kmean, s.dvar, seq_after[t], sel, n_sel, blk_logit, None,
                              ws)
        P.compkv_sparse_decode(dims, scale, Q[L][t], Ks[L], Vs[L], s.vmean, blk_logit, seq_after[t], sel, n_sel,
                               out, lse, ws)

    def dense(L, t):
        Ks[L][:, :, n0 + t] = Kn[L][t]
        Vs[L][:, :, n0 + t] = Vn[L][t]
        P.compkv_dense_decode(dims, scale, Q[L][t], Ks[L], Vs[L], seq_after[t], out, lse, ws)

    def per_step_us(fn):
        """Per-step times (us per step, all layers) of a pass over every step, after a warm-up pass."""
        graphs = []
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):  # eager warm-up of the launch path off the capture
            for L in range(Lyr):
                fn(L, 0)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        for t in range(T):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for L in range(Lyr):
                    fn(L, t)
            graphs.append(g)
        for g in graphs:
            g.replay()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(T + 1)]
        ev[0].record()
        for t, g in enumerate(graphs):
            g.replay()
            ev[t + 1].record()
        torch.cuda.synchronize()
        return [ev[t].elapsed_time(ev[t + 1]) * 1e3 for t in range(T)]

    wall0 = time.perf_counter()
    us_sep = per_step_us(separate)
    us_dense = per_step_us(dense)
    us = per_step_us(fused)  # last, so the outputs below are the fused step's
    wall = time.perf_counter() - wall0
    torch.cuda.synchronize()
    X_last = -(-(n0 + T) // w.block_size)
    nsel_host = n_sel.cpu().numpy().reshape(-1)
    assert np.all(nsel_host == min(budget, X_last)), "selection count mismatch"
    sel_host = sel.cpu().numpy().reshape(-1, budget)
    sel_lists = [list(sel_host[u, :nsel_host[u]]) for u in range(w.units)]

    win = slice(193, 209)
    per_layer = np.array(us) / Lyr
    ab = algorithmic_bytes(w.with_(context=n0 + T), budget, sel_lists)
    step_bytes = ab["score_select"] + ab["sparse_decode"] + ab["append_stats"]
    mean_us = float(per_layer.mean())
    ach = step_bytes / (mean_us * 1e-6) / 1e9
    line = {
        "metric": "us/decode-step/layer and HBM GB/s (fraction of peak); speedup vs dense decode",
        "unit": "us/decode-step/layer",
        "value": round(mean_us, 3),
        "n_gpus": 1,
        "steps": T,
        "warmup": T,
        "ms_per_step": round(float(np.mean(us)) / 1e3, 6),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 K/V/q, fp32 summaries and accumulation",
        "data": "synthetic (seeded block-structured keys, N(0,1) values, fresh N(0,1)/sqrt(128) queries per step)",
        "config": {"workload": w.name, "batch": w.batch, "n_q_heads": w.n_q_heads, "n_kv_heads": w.n_kv_heads,
                   "head_dim": w.head_dim, "prefill": n0, "decode_steps": T, "layers": Lyr,
                   "block_size": w.block_size, "budget_blocks": budget, "n_var_groups": w.n_var_groups,
                   "parallelism": "single GPU"},
        "value_steps_193_208": round(float(per_layer[win].mean()), 3),
        "sd_us": round(float(per_layer.std(ddof=1)), 3),
        "separate_calls_us_per_step": round(float(np.mean(us_sep)) / Lyr, 3),
        "dense_us_per_step": round(float(np.mean(us_dense)) / Lyr, 3),
        "speedup_vs_dense": round(float(np.mean(us_dense)) / float(np.mean(us)), 3),
        "hbm_gbps": round(ach, 1),
        "hbm_frac": round(ach / HBM_PEAK_GBPS, 4),
        "algorithmic_bytes_per_step": step_bytes,
        "roofline": {"kernel": step_kernels(P.compkv_decode_step_path(dims, params)), "bound": "hbm",
                     "achieved": round(ach, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBPS, 4),
                     "traffic": measured_traffic(w.name, "decode_step"),
                     "algorithmic_bytes_per_launch": step_bytes},
        "wall_s": round(wall, 2),
    }
    if not args.no_cpu_baseline:
        Kb, Vb = host0
        wq = w.with_(context=n0)
        qb = np.stack([gen_queries(w, 0, b, 0) for b in range(w.batch)])
        line["cpu_baseline"] = cpu_baseline(wq, budget, Kb, Vb, qb, args.cpu_seconds)
    print(json.dumps(line), flush=True)



def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the path shards by KV head "
              "with no exchange, so per-GPU work is the single-GPU step)", file=sys.stderr)
        sys.exit(2)
    import torch

    if args.copy_calibration:
        src = torch.empty(args.copy_calibration << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": src.numel(), "copies": 3}))
        return

    import paper_2609_26300_amd as P
    from workloads import WORKLOADS, gen_layer

    w = WORKLOADS[args.workload]
    if args.n_var_groups:
        w = w.with_(n_var_groups=args.n_var_groups)
    if args.context:
        w = w.with_(context=args.context, name=f"{w.name} at {args.context} tokens")
    if w.decode_steps > 0:
        return run_streaming(args, w)
    budget = args.budget or w.budget_blocks
    dev = "cuda"
    scale = 1.0 / math.sqrt(w.head_dim)
    n = w.context
    Kb, Vb, qb = gen_layer(w, 0)
    layer_bytes = Kb.nbytes * 2
    layers = args.layers or max(4, min(32, math.ceil(1.2e9 / layer_bytes)))

    def to_dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(dev)

    dims = P.make_dims(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.block_size, w.n_var_groups,
                       w.capacity, max_seq_len=n)
    K0, V0 = to_dev(Kb), to_dev(Vb)
    q = to_dev(qb)
    k_new = K0[:, :, n - 1].contiguous()
    v_new = V0[:, :, n - 1].contiguous()
    page = args.page_tokens
    if page:  # the same cache scattered over randomly permuted pages
        pps = -(-w.capacity // page)
        perm = np.random.default_rng(0).permutation(w.batch * pps).reshape(w.batch, pps).astype(np.int32)
        table = torch.from_numpy(perm).to(dev)
        dims = P.make_dims(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.block_size, w.n_var_groups,
                           pps * page, max_seq_len=n, block_table=table, page_tokens=page, num_pages=w.batch * pps)
        dest = torch.from_numpy(perm.reshape(-1)).long().to(dev)

        def paged(X):
            Xc = torch.zeros((w.batch, w.n_kv_heads, pps * page, w.head_dim), dtype=X.dtype, device=dev)
            Xc[:, :, :X.shape[2]] = X
            Xv = Xc.view(w.batch, w.n_kv_heads, pps, page, w.head_dim).permute(0, 2, 1, 3, 4)
            out = torch.empty((w.batch * pps, w.n_kv_heads, page, w.head_dim), dtype=X.dtype, device=dev)
            out[dest] = Xv.reshape(w.batch * pps, w.n_kv_heads, page, w.head_dim)
            return out

        K0, V0 = paged(K0), paged(V0)
        torch.cuda.synchronize()
    seq_before = torch.full((w.batch,), n - 1, dtype=torch.int32, device=dev)
    seq_after = torch.full((w.batch,), n, dtype=torch.int32, device=dev)
    Ks, Vs, summ = [], [], []
    for layer in range(layers):
        K = K0 if layer == 0 else K0.clone()
        V = V0 if layer == 0 else V0.clone()
        s = P.alloc_summaries(dims)
        P.compkv_build_stats(dims, K, V, seq_after, s.kmean, s.dvar, s.vmean)
        if args.host_kv:  # the layer's cache moves to pinned host memory
            K = torch.empty(K.shape, dtype=K.dtype, pin_memory=True).copy_(K)
            V = torch.empty(V.shape, dtype=V.dtype, pin_memory=True).copy_(V)
            if args.host_summaries:  # and its summaries
                for f in ("kmean", "dvar", "vmean"):
                    x = getattr(s, f)
                    setattr(s, f, torch.empty(x.shape, dtype=x.dtype, pin_memory=True).copy_(x))
        Ks.append(K)
        Vs.append(V)
        summ.append(s)
    if args.host_kv:
        K0 = V0 = None
        torch.cuda.empty_cache()
    units = (w.batch, w.n_kv_heads)
    ws = P.alloc_workspace(dims, budget)
    sel = torch.empty((*units, budget), dtype=torch.int32, device=dev)
    n_sel = torch.empty(units, dtype=torch.int32, device=dev)
    blk_logit = torch.empty((*units, w.group, dims.xcap), dtype=torch.float32, device=dev)
    out = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=torch.float32, device=dev)
    lse = torch.empty((w.batch, w.n_q_heads), dtype=torch.float32, device=dev)
    path = {"auto": P.COMPKV_SELECT_AUTO, "chunked": P.COMPKV_SELECT_CHUNKED,
            "one_group": P.COMPKV_SELECT_ONE_GROUP, "chunked_exact": P.COMPKV_SELECT_CHUNKED_EXACT,
            "stream": P.COMPKV_SELECT_STREAM}[args.select_path]
    kind = {"compkv": P.COMPKV_SCORE_COMPKV, "mass": P.COMPKV_SCORE_MASS,
            "first_order": P.COMPKV_SCORE_FIRST_ORDER}[args.score_kind]
    drop = args.compensation == "drop"
    params = P.CompkvSelectParams(budget, 1, 2, scale, path, kind, P.COMPKV_COMP_DROP if drop else P.COMPKV_COMP_MEAN)
    step_path = P.compkv_decode_step_path(dims, params)
    torch.cuda.synchronize()

    def append(L):
        s = summ[L]
        P.compkv_append_stats(dims, Ks[L], Vs[L], k_new, v_new, seq_before, s.kmean, s.dvar, s.vmean)

    def score(L):
        s = summ[L]
        P.compkv_score_select(dims, params, q, s.kmean, s.dvar, seq_after, sel, n_sel, blk_logit, None, ws)

    def decode(L):
        P.compkv_sparse_decode(dims, scale, q, Ks[L], Vs[L], None if drop else summ[L].vmean,
                               None if drop else blk_logit, seq_after, sel, n_sel, out, lse, ws)

    def fused(L):
        s = summ[L]
        P.compkv_decode_step(dims, params, q, Ks[L], Vs[L], k_new, v_new, seq_after, s.kmean, s.dvar, s.vmean,
                             sel, n_sel, blk_logit, None, out, lse, ws)

    def row_write(L):
        if args.host_kv:  # (a host cache row is not written inside torch's captured graphs)
            return
        if page:
            for b in range(w.batch):
                pg, r = int(perm[b, (n - 1) // page]), (n - 1) % page
                Ks[L][pg, :, r] = k_new[b]
                Vs[L][pg, :, r] = v_new[b]
        else:
            Ks[L][:, :, n - 1] = k_new
            Vs[L][:, :, n - 1] = v_new

    def dense(L):
        P.compkv_dense_decode(dims, scale, q, Ks[L], Vs[L], seq_after, out, lse, ws)

    def capture(fns, layer_ids):
        """One HIP graph running fns (in order) for each layer in layer_ids."""
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):  # eager warm-up off the capture
            for L in layer_ids:
                for f in fns:
                    f(L)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for L in layer_ids:
                for f in fns:
                    f(L)
        torch.cuda.synchronize()
        return g

    def run_steps(fns, steps, warmup):
        """Time exactly `steps` steps (one layer each, rotating) as replays of captured graphs."""
        if args.eager:
            for i in range(warmup):
                for f in fns:
                    f(i % layers)
            torch.cuda.synchronize()
            t0 = torch.cuda.Event(enable_timing=True)
            t1 = torch.cuda.Event(enable_timing=True)
            wall0 = time.perf_counter()
            t0.record()
            for i in range(steps):
                for f in fns:
                    f(i % layers)
            t1.record()
            torch.cuda.synchronize()
            return t0.elapsed_time(t1) * 1e3 / steps, time.perf_counter() - wall0
        full = capture(fns, list(range(layers)))
        tail_n = steps % layers
        tail = capture(fns, list(range(tail_n))) if tail_n else None

        def replay(k):
            for _ in range(k // layers):
                full.replay()
            if k % layers:
                (tail if k % layers == tail_n else capture(fns, list(range(k % layers)))).replay()

        replay(warmup)
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        wall0 = time.perf_counter()
        t0.record()
        replay(steps)
        t1.record()
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) * 1e3 / steps, time.perf_counter() - wall0

    def step_samples(fns, steps):
        """Per-step times (us): one captured graph per layer, each replay followed by an event on the
        launch stream, so consecutive events bracket exactly one step."""
        graphs = [capture(fns, [L]) for L in range(layers)]
        for i in range(min(steps, 2 * layers)):
            graphs[i % layers].replay()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        ev[0].record()
        for i in range(steps):
            graphs[i % layers].replay()
            ev[i + 1].record()
        torch.cuda.synchronize()
        return np.array([ev[i].elapsed_time(ev[i + 1]) * 1e3 for i in range(steps)])

    def fused_at(K):
        """The fused step at budget K with its own selection outputs and workspace."""
        pk = P.CompkvSelectParams(K, 1, 2, scale, path, kind, params.compensation)
        wk = P.alloc_workspace(dims, K)
        sk = torch.empty((*units, K), dtype=torch.int32, device=dev)

        def f(L):
            s = summ[L]
            P.compkv_decode_step(dims, pk, q, Ks[L], Vs[L], k_new, v_new, seq_after, s.kmean, s.dvar, s.vmean,
                                 sk, n_sel, blk_logit, None, out, lse, wk)
        return f, pk, sk

    result = {}
    if args.only in ("all", "sparse", "fused"):
        us, wall = run_steps([fused], args.steps, args.warmup)
        samples = None if args.eager else step_samples([fused], args.steps)
        us_sep, per_k = None, {}
        if args.only != "fused":
            us_sep, _ = run_steps([append, score, decode], args.steps, args.warmup)
            per_k = {name: run_steps([f], args.steps, args.warmup)[0]
                     for name, f in (("append_stats", append), ("score_select", score), ("sparse_decode", decode))}
        # leave the outputs of a complete step for the checks below
        fused(0)
        torch.cuda.synchronize()
        result["sparse"] = (us, per_k, wall, us_sep, samples)
        sel_host = sel.cpu().numpy().reshape(-1, budget)
        nsel_host = n_sel.cpu().numpy().reshape(-1)
        sel_lists = [list(sel_host[u, :nsel_host[u]]) for u in range(w.units)]
        assert all(len(s) == min(budget, -(-n // w.block_size)) for s in sel_lists), "selection count mismatch"
        sweep = []
        if args.only == "all" and not args.no_sweep and args.budget is None:
            for K in BUDGET_SWEEPS.get(w.name, ()):
                if K == budget:
                    continue
                f, pk, sk = fused_at(K)
                us_k, _ = run_steps([f], args.steps, args.warmup)
                f(0)
                torch.cuda.synchronize()
                sh, nh = sk.cpu().numpy().reshape(-1, K), n_sel.cpu().numpy().reshape(-1)
                lists = [list(sh[u, :nh[u]]) for u in range(w.units)]
                ab_k = algorithmic_bytes(w, K, lists, not drop)
                b_k = ab_k["score_select"] + ab_k["sparse_decode"] + ab_k["append_stats"]
                sweep.append(dict(budget_blocks=K, us=round(us_k, 3), algorithmic_bytes=b_k,
                                  hbm_frac=round(b_k / (us_k * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                                  select_path=PATH_NAMES[P.compkv_decode_step_path(dims, pk)]))
            fused(0)
            torch.cuda.synchronize()
    if args.only in ("all", "dense"):
        us_d, wall_d = run_steps([row_write, dense], args.steps, args.warmup)
        per_kd = {"dense_decode": run_steps([dense], args.steps, args.warmup)[0]}
        result["dense"] = (us_d, per_kd, wall_d)

    line = {
        "metric": "us/decode-step/layer and HBM GB/s (fraction of peak); speedup vs dense decode",
        "unit": "us/decode-step/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 K/V/q, fp32 summaries and accumulation",
        "data": "synthetic (seeded block-structured keys, N(0,1) values, N(0,1)/sqrt(128) queries)",
        "config": {"workload": w.name, "batch": w.batch, "n_q_heads": w.n_q_heads, "n_kv_heads": w.n_kv_heads,
                   "head_dim": w.head_dim, "context": n, "block_size": w.block_size, "budget_blocks": budget,
                   "n_var_groups": w.n_var_groups, "layer_copies": layers, "parallelism": "single GPU",
                   "select_path": PATH_NAMES[step_path], "score_kind": args.score_kind,
                   "compensation": args.compensation, "page_tokens": page,
                   "kv_memory": "pinned host" if args.host_kv else "device",
                   "summary_memory": "pinned host" if args.host_kv and args.host_summaries else "device"},
    }
    if "sparse" in result:
        us, per_k, wall, us_sep, samples = result["sparse"]
        ab = algorithmic_bytes(w, budget, sel_lists, not drop)
        step_bytes = ab["score_select"] + ab["sparse_decode"] + ab["append_stats"]
        ach = step_bytes / (us * 1e-6) / 1e9
        line.update({
            "value": round(us, 3),
            "ms_per_step": round(us / 1e3, 6),
            "hbm_gbps": round(ach, 1),
            "hbm_frac": round(ach / HBM_PEAK_GBPS, 4),
            "algorithmic_bytes_per_step": step_bytes,
            # mean and sample SD over individually timed steps (one graph replay per step)
            "step_us_mean": round(float(samples.mean()), 3) if samples is not None else None,
            "step_us_sd": round(float(samples.std(ddof=1)), 3) if samples is not None else None,
            "separate_calls_us_per_step": round(us_sep, 3) if us_sep is not None else None,
            "separate_call_us": {k: round(v, 3) for k, v in per_k.items()},
            # the timed call: its dispatches are the whole step
            "roofline": {"kernel": step_kernels(step_path), "bound": "hbm",
                         "achieved": round(ach, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                         "frac": round(ach / HBM_PEAK_GBPS, 4), "traffic": measured_traffic(w.name, "decode_step"),
                         "algorithmic_bytes_per_launch": step_bytes},
        })
    if "sparse" in result and sweep:
        line["budget_sweep"] = sweep + [dict(budget_blocks=budget, us=line["value"],
                                             algorithmic_bytes=line["algorithmic_bytes_per_step"],
                                             hbm_frac=line["hbm_frac"], select_path=PATH_NAMES[step_path])]
        line["budget_sweep"].sort(key=lambda e: e["budget_blocks"])
    if "dense" in result:
        us_d, per_kd, _ = result["dense"]
        line["dense_us_per_step"] = round(us_d, 3)
        line["dense_kernel_us"] = {k: round(v, 3) for k, v in per_kd.items()}
        if "sparse" in result:
            line["speedup_vs_dense"] = round(us_d / line["value"], 3)
            for e in line.get("budget_sweep", []):
                e["speedup_vs_dense"] = round(us_d / e["us"], 3)
            ab_d = algorithmic_bytes(w, budget, sel_lists)["dense_decode"]
            line["dense_hbm_gbps"] = round(ab_d / (per_kd["dense_decode"] * 1e-6) / 1e9, 1)
    if not args.host_kv and not page:  # the prefill (compkv_build_stats) of one layer, outside the step
        for _ in range(2):
            P.compkv_build_stats(dims, Ks[0], Vs[0], seq_after, summ[0].kmean, summ[0].dvar, summ[0].vmean)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(5):
            P.compkv_build_stats(dims, Ks[0], Vs[0], seq_after, summ[0].kmean, summ[0].dvar, summ[0].vmean)
        e1.record()
        torch.cuda.synchronize()
        us_b = e0.elapsed_time(e1) * 1e3 / 5
        X = -(-n // w.block_size)
        b_bytes = (w.batch * w.n_kv_heads * (n * w.head_dim * 2 * 2 + X * (2 * w.head_dim + w.n_var_groups) * 4))
        line["prefill_build_us"] = round(us_b, 1)
        line["prefill_hbm_gbps"] = round(b_bytes / (us_b * 1e-6) / 1e9, 1)
    line["paper_context"] = ("paper: up to 6.85x self-attention speedup over full attention, CPU-offload "
                             "pipeline on one NVIDIA H100 80GB + 4 host threads, PCIe-bound (128K, 512-token "
                             "budget); not comparable with an HBM-resident MI355X step")
    if not args.no_cpu_baseline and "sparse" in result:
        line["cpu_baseline"] = cpu_baseline(w, budget, Kb, Vb, qb, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
