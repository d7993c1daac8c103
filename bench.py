#!/usr/bin/env python3
"""Benchmark of the relaxed online long convolution on one MI355X.

One "step" is one whole online generation: reset, then L positions of
lcsm_step for all M layers (red cells and batched gray tiles), with the
teacher-forced inputs already resident in HBM.  The metric is mixer
tokens/s = B * L / (seconds per step).

Printed: one JSON line (see --help), with a roofline entry for the kernel
that takes the largest share of the GPU time (per-launch durations measured
with HIP events in a separate pass over the same kernels) and the CPU oracle
timed on a bounded sample of the same workload.
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
DEFAULT_WORKLOAD = "m1b8d768l8k"


def parse():
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=4)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--workload", default=DEFAULT_WORKLOAD)
    p.add_argument("--direct-max-u", type=int, default=0, help="0 = library default")
    p.add_argument("--lds-fft-max-n", type=int, default=0, help="0 = library default")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-budget", type=float, default=20.0, help="seconds of oracle work, about")
    p.add_argument("--no-kernel-pass", action="store_true")
    p.add_argument("--closed-loop", action="store_true", help="also time the tanh-chain generation")
    return p.parse_args()


# ----------------------------------------------------------------- algorithmic bytes
def tile_bytes(kind, U, w, fused):
    """Algorithmic HBM bytes of one launch, for all M layers.

    Per column (m, b, d): red cell 16 B (read y_t and acc_t, write z_t and the
    slot); gray tile: read the U-input window (4U; U-1 of it when the red
    cell is fused and y_t comes from the register) and read+write the U
    destination accumulators (8U).  Per (m, d): the lags 1..2U-1 (4(2U-1))
    for a direct tile, or the U+1 complex bins of the cached spectrum (8(U+1))
    for an FFT tile."""
    cols = w.M * w.B * w.D
    md = w.M * w.D
    if kind == "red":
        return 16 * cols
    if kind == "fused":
        return 16 * cols + (4 * (U - 1) + 8 * U) * cols + 4 * (2 * U - 1) * md
    if kind == "direct":
        return (12 * U) * cols + 4 * (2 * U - 1) * md
    return (12 * U) * cols + 8 * (U + 1) * md


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(the library has no multi-GPU path).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import datagen
    import paper_2410_12982_amd.lcsm as lcsm

    w = datagen.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    opts = {}
    if args.direct_max_u:
        opts["direct_max_u"] = args.direct_max_u
    if args.lds_fft_max_n:
        opts["lds_fft_max_n"] = args.lds_fft_max_n
    opts = opts or None

    print(f"# workload {w.name}: M={w.M} B={w.B} D={w.D} L={w.L}", file=sys.stderr, flush=True)
    filters = datagen.filters_torch(w, dev)
    y = datagen.y_torch(w, dev)                      # [L, M, B, D] resident in HBM
    z = torch.empty_like(y)
    ctx = lcsm.Lcsm(filters, w.B, options=opts)
    torch.cuda.synchronize()

    def one_step():
        ctx.reset()
        ctx.run(y, z)

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    print(f"# warmup done ({args.warmup})", file=sys.stderr, flush=True)

    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    ev0.record()
    for _ in range(args.steps):
        one_step()
    ev1.record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms = ev0.elapsed_time(ev1) / args.steps
    value = w.B * w.L / (ms / 1e3)
    print(f"# timed {args.steps} steps: {ms:.3f} ms/step (wall {1e3 * t_wall / args.steps:.3f})",
          file=sys.stderr, flush=True)

    # ---------------------------------------------------------- per-kernel pass
    roofline = None
    levels = {}
    if not args.no_kernel_pass:
        roofline, levels = kernel_pass(ctx, w, y, z, opts, lcsm, torch)

    closed = None
    if args.closed_loop:
        x = datagen.x_torch(w, dev)
        torch.cuda.synchronize()
        ctx.reset()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for t in range(w.L):
            ctx.step_chain(x[t], z[t])
        e1.record()
        torch.cuda.synchronize()
        cms = e0.elapsed_time(e1)
        closed = {"ms": round(cms, 3), "tokens_per_s": w.B * w.L / (cms / 1e3)}
        del x

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, args.cpu_budget)

    out = {
        "metric": "mixer tokens/s (B*L/s)",
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded counter-based generator; teacher-forced inputs resident in HBM)",
        "config": {"workload": w.name, "M": w.M, "B": w.B, "D": w.D, "L": w.L,
                   "options": opts or "default", "parallelism": "single-gpu"},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    if levels:
        out["per_level_us"] = levels
    if closed:
        out["closed_loop"] = closed
    print(json.dumps(out), flush=True)
    ctx.close()


def kernel_pass(ctx, w, y, z, opts, lcsm, torch):
    """Per-launch durations by tile level, with HIP events on the context's
    stream.  Steps whose tile is fused into the red-cell kernel are one
    launch; other steps are driven as red cells (lcsm_step_layer) followed by
    the tile launch alone (lcsm_advance), bracketed by events."""
    stream = torch.cuda.current_stream()
    L = w.L
    plans = [ctx.plan(t) for t in range(L)]
    ctx.reset()
    recs = []
    pool = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in range(min(L, 4096))]
    k = 0
    for t in range(L):
        i, U, n, kind = plans[t]
        fused = kind == lcsm.TILE_DIRECT and U <= 32 or kind == lcsm.TILE_NONE
        a, b = pool[k % len(pool)]
        if fused:
            a.record(stream)
            ctx.step(y[t], z[t])
            b.record(stream)
            recs.append(("fused" if U else "red", U, kind, a, b))
        else:
            for m in range(w.M):
                ctx.step_layer(m, y[t, m], z[t, m])
            a.record(stream)
            ctx.advance()
            b.record(stream)
            recs.append((lcsm.TILE_KIND_NAMES[kind], U, kind, a, b))
        k += 1
        if k % len(pool) == 0:
            torch.cuda.synchronize()
            recs = _harvest(recs)
    torch.cuda.synchronize()
    recs = _harvest(recs)
    # aggregate by (kernel, U)
    agg = {}
    for name, U, kind, dur in recs:
        key = (name, U)
        s = agg.setdefault(key, [0.0, 0])
        s[0] += dur
        s[1] += 1
    levels = {f"{name}:U={U}": {"launches": n, "avg_us": round(1e3 * tot / n, 3),
                                "total_ms": round(tot, 3)}
              for (name, U), (tot, n) in sorted(agg.items(), key=lambda kv: kv[0][1])}
    (name, U), (tot, n) = max(agg.items(), key=lambda kv: kv[1][0])
    avg_s = tot / n / 1e3
    fused = name == "fused"
    kind_for_bytes = "fused" if fused else ("red" if name == "red" else
                                            ("direct" if name == "direct" else "fft"))
    nbytes = tile_bytes(kind_for_bytes, U, w, fused)
    achieved = nbytes / avg_s / 1e9
    roofline = {"bound": "hbm", "kernel": f"{name} tile U={U}", "achieved": round(achieved, 2),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 5),
                "traffic": None, "bytes_per_launch": nbytes, "avg_launch_us": round(avg_s * 1e6, 3),
                "share_of_gpu_time": round(tot / sum(v[0] for v in agg.values()), 4)}
    return roofline, levels


def _harvest(recs):
    out = []
    for r in recs:
        if len(r) == 5:
            name, U, kind, a, b = r
            out.append((name, U, kind, a.elapsed_time(b)))
        else:
            out.append(r)
    return out


def cpu_baseline(w, budget_s):
    """Time the CPU oracle (relaxed tiling, fp64 numpy, as it stands) on a
    bounded sample: all positions of a subset of (b, d) columns of layer 0,
    with the sample size grown until about budget_s seconds of work."""
    import numpy as np

    import datagen
    from oracle import feedback
    from oracle.relaxed import relaxed_online

    total_cols = w.M * w.B * w.D
    ncols = 8
    elapsed = 0.0
    while True:
        d_idx = np.arange(min(ncols, w.D))
        b_idx = np.arange(max(1, min(w.B, ncols // len(d_idx))))
        n = len(d_idx) * len(b_idx)
        h = datagen.filters_np(w, m_idx=[0], d_idx=d_idx)[0]          # [n_d, L]
        hc = np.broadcast_to(h.T[:, None, None, :], (w.L, 1, len(b_idx), len(d_idx)))
        hc = np.ascontiguousarray(hc).reshape(w.L, 1, n)
        yc = datagen.y_np(w, m_idx=[0], b_idx=b_idx, d_idx=d_idx).reshape(w.L, 1, n)
        t0 = time.perf_counter()
        relaxed_online(hc, feedback.teacher_forced(yc))
        elapsed = time.perf_counter() - t0
        if elapsed * 4 > budget_s or n >= total_cols or ncols >= 8192:
            break
        ncols *= 4
    # tokens/s over the whole workload: B*L tokens need total_cols columns
    per_col_s = elapsed / n
    value = w.B * w.L / (per_col_s * total_cols)
    return {"value": round(value, 2), "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": f"relaxed-tiling oracle (fp64 numpy), all {w.L} positions of {n} of "
                      f"{total_cols} columns in {elapsed:.1f} s, scaled linearly to all columns"}


if __name__ == "__main__":
    main()
