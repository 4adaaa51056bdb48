"""Phase breakdown of the fused decode step from the library's phase-trace build.

    python -m paper_2609_26300_amd.phase_trace --workload long_128k [--steps 8] [--build]

Runs compkv_decode_step on the chunked-exact launch shape (the chunk-scoring launch, then the fused
selection/exact launch) over resident layer copies of a synthetic workload, with libcompkv_trace.so
(built by paper_2609_26300_amd/build.py with trace=True; --build rebuilds it first) in place of
libcompkv.so. Every workgroup's thread 0 stamps the GPU's 100 MHz real-time counter at its phase
boundaries (compkv_phase_trace_set); this prints, per launch and workgroup role, the phase durations
(percentiles over workgroups and steps, microseconds) and the critical path of the step, as markdown.
The marks add a few instructions per phase and leave every kernel's occupancy as in the normal build;
the time per step with the trace on and off is reported beside the records.
"""
from __future__ import annotations

import argparse
import math
import os
import sys

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

TICK_US = 0.01  # the real-time counter runs at 100 MHz

# (label, from slot, to slot) per launch and role; slot 15 is the workgroup's end
CHUNK_PHASES = {
    1: ("chunk workgroups", [("query in LDS", 0, 2), ("first slot of blocks", 2, 3), ("remaining slots", 3, 4),
                             ("partials formed", 4, 6), ("stores", 6, 15), ("whole", 0, 15)]),
    2: ("last-block workgroups", [("whole", 0, 15)]),
}
FUSED_PHASES = {
    1: ("selecting workgroups", [("selection loads", 0, 2), ("normalizers and keys", 2, 3), ("top-K", 3, 4),
                                 ("exact tiles (wave 0)", 4, 8), ("partial", 8, 9), ("arrival and merge", 9, 15),
                                 ("whole", 0, 15)]),
    2: ("streaming workgroups", [("weights formed", 0, 5), ("mean values streamed", 5, 6), ("ids in hand", 6, 7),
                                 ("exact tiles (wave 0)", 7, 8), ("partial", 8, 9), ("arrival and merge", 9, 15),
                                 ("whole", 0, 15)]),
}


def _pct(x):
    return " | ".join(f"{v:.2f}" for v in np.percentile(x, [10, 50, 90, 100]))


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", default="long_128k")
    ap.add_argument("--steps", type=int, default=8, help="traced steps (one layer copy each)")
    ap.add_argument("--build", action="store_true", help="rebuild libcompkv_trace.so first")
    args = ap.parse_args(argv)

    from paper_2609_26300_amd import build as lib_build

    if args.build or not os.path.exists(lib_build.TRACE_LIB):
        lib_build.build(trace=True)
    import paper_2609_26300_amd.binding as B

    B.LIB_PATH = lib_build.TRACE_LIB  # before the first call loads a library
    import torch

    import paper_2609_26300_amd as P
    from workloads import WORKLOADS, gen_layer

    w = WORKLOADS[args.workload]
    n = w.context
    Kb, Vb, qb = gen_layer(w, 0)
    dev = torch.device("cuda:0")

    def up(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(dev)

    dims = P.make_dims(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.block_size, w.n_var_groups, w.capacity,
                       max_seq_len=n)
    layers = max(4, math.ceil(1.2e9 / (Kb.nbytes * 2)))  # more than the last-level cache holds
    K0, V0 = up(Kb), up(Vb)
    Ks = [K0] + [K0.clone() for _ in range(layers - 1)]
    Vs = [V0] + [V0.clone() for _ in range(layers - 1)]
    q = up(qb)
    k_new = K0[:, :, n - 1].contiguous()
    v_new = V0[:, :, n - 1].contiguous()
    sl = torch.full((w.batch,), n, dtype=torch.int32, device=dev)
    summ = []
    for L in range(layers):
        s = P.alloc_summaries(dims, dev)
        P.compkv_build_stats(dims, Ks[L], Vs[L], sl, s.kmean, s.dvar, s.vmean)
        summ.append(s)
    Kbud = w.budget_blocks
    units = (w.batch, w.n_kv_heads)
    ws = P.alloc_workspace(dims, Kbud, dev)
    sel = torch.empty((*units, Kbud), dtype=torch.int32, device=dev)
    nsel = torch.empty(units, dtype=torch.int32, device=dev)
    blk = torch.empty((*units, w.group, dims.xcap), dtype=torch.float32, device=dev)
    out = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=torch.float32, device=dev)
    lse = torch.empty((w.batch, w.n_q_heads), dtype=torch.float32, device=dev)
    prm = P.CompkvSelectParams(Kbud, 1, 2, 1.0 / math.sqrt(w.head_dim), P.COMPKV_SELECT_CHUNKED_EXACT)

    def step(L):
        s = summ[L]
        P.compkv_decode_step(dims, prm, q, Ks[L], Vs[L], k_new, v_new, sl, s.kmean, s.dvar, s.vmean, sel, nsel, blk,
                             None, out, lse, ws)

    for i in range(3 * layers):
        step(i % layers)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(nsteps):
        ev0.record()
        for i in range(nsteps):
            step(i % layers)
        ev1.record()
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) * 1e3 / nsteps

    untraced_us = timed(4 * layers)
    words = 1 << 20  # 16 words per workgroup: up to 65536 workgroups per launch
    rec1 = torch.zeros(words, dtype=torch.int64, device=dev)
    rec2 = torch.zeros(words, dtype=torch.int64, device=dev)
    P.compkv_phase_trace_set(rec1, rec2)
    traced_us = timed(4 * layers)  # every step overwrites the records
    chunks, fused = [], []
    for i in range(args.steps):
        rec1.zero_()
        rec2.zero_()
        torch.cuda.synchronize()
        step(i % layers)
        torch.cuda.synchronize()
        a = rec1.cpu().numpy().view(np.uint64).reshape(-1, 16)
        b = rec2.cpu().numpy().view(np.uint64).reshape(-1, 16)
        a, b = a[a[:, 15] != 0], b[b[:, 15] != 0]
        t0 = int(a[:, 0].min())

        def rel(x, t0=t0):
            return (x.astype(np.int64) - t0) * TICK_US

        chunks.append((a, rel))
        fused.append((b, rel))
    P.compkv_phase_trace_set(None, None)

    lines = [f"# Phase breakdown of the fused step: {args.workload}", "",
             "Command (paths relative to the repository root):", "", "```",
             f"python -m paper_2609_26300_amd.phase_trace --workload {args.workload} --steps {args.steps}", "```", "",
             f"Layer copies: {layers}; budget {Kbud} blocks; launch shape chunked_exact "
             f"({'one selector per unit' if np.any([np.any(f[0][:, 7] != 0) for f in fused]) else 'item and compensation workgroups'}).",
             f"Events around {4 * layers} back-to-back steps of the trace library: {untraced_us:.2f} us per step recording nothing, "
             f"{traced_us:.2f} recording. The records below are of {args.steps} single steps (one layer copy each),",
             "each started on an idle GPU.", "",
             "Times in microseconds from the chunk launch's first workgroup start (GPU real-time counter, 100 MHz),",
             "percentiles p10 | p50 | p90 | max over workgroups and steps.", ""]

    def table(title, recs, phases):
        lines.extend([f"## {title}", ""])
        for role, (name, ph) in phases.items():
            rows = [np.concatenate([r[r[:, 1] == role] for r, _ in recs])]
            m = rows[0]
            if len(m) == 0:
                continue
            cnt = len(m) // len(recs)
            lines.extend([f"{name} ({cnt} per step)", "", "| phase | p10 | p50 | p90 | max |", "|---|---|---|---|---|"])
            for label, s0, s1 in ph:
                ok = (m[:, s0] != 0) & (m[:, s1] != 0)
                if ok.sum() == 0:
                    continue
                d = (m[ok, s1].astype(np.int64) - m[ok, s0].astype(np.int64)) * TICK_US
                lines.append(f"| {label} | {_pct(d)} |")
            st = np.concatenate([rel(r[r[:, 1] == role][:, 0]) for r, rel in recs])
            en = np.concatenate([rel(r[r[:, 1] == role][:, 15]) for r, rel in recs])
            lines.extend([f"| start (from step start) | {_pct(st)} |", f"| end (from step start) | {_pct(en)} |", ""])

    def by_xcd(title, recs):
        # end times of each XCD's workgroups (slot 14 holds the XCC id in its high word)
        ends = {}
        for r, rel in recs:
            x = (r[:, 14] >> np.uint64(32)).astype(np.int64)
            for xcd in np.unique(x):
                ends.setdefault(int(xcd), []).append(rel(r[x == xcd][:, 15]))
        lines.extend([f"{title}: workgroup end times per XCD", "", "| XCD | workgroups per step | p10 | p50 | p90 | max |",
                      "|---|---|---|---|---|---|"])
        for xcd in sorted(ends):
            e = np.concatenate(ends[xcd])
            lines.append(f"| {xcd} | {len(e) // len(recs)} | {_pct(e)} |")
        lines.append("")

    table("Chunk-scoring launch", chunks, CHUNK_PHASES)
    by_xcd("Chunk-scoring launch", chunks)
    table("Fused selection/exact launch", fused, FUSED_PHASES)
    by_xcd("Fused selection/exact launch", fused)
    # the step's critical path, median over steps
    k1_end = np.median([rel(r[:, 15]).max() for r, rel in chunks])
    k2_start = np.median([rel(r[:, 0]).min() for r, rel in fused])
    k2_end = np.median([rel(r[:, 15]).max() for r, rel in fused])
    sel_end = np.median([rel(r[r[:, 1] == 1][:, 4]).max() for r, rel in fused])
    stream_end = [rel(r[r[:, 1] == 2][:, 6]) for r, rel in fused]
    stream_end = np.median([x.max() for x in stream_end if len(x)]) if any(len(x) for x in stream_end) else float("nan")
    merge_start = np.median([rel(r[r[:, 10] != 0][:, 10]).max() for r, rel in fused])
    lines.extend(["## Critical path (medians over steps)", "",
                  "| event | us from step start |", "|---|---|",
                  f"| last chunk-launch workgroup ends | {k1_end:.2f} |",
                  f"| first fused-launch workgroup starts | {k2_start:.2f} |",
                  f"| last selection done | {sel_end:.2f} |",
                  f"| last mean values weighed | {stream_end:.2f} |",
                  f"| last merge starts | {merge_start:.2f} |",
                  f"| last fused-launch workgroup ends | {k2_end:.2f} |", ""])
    print("\n".join(lines))


if __name__ == "__main__":
    main()
