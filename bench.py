#!/usr/bin/env python3
"""Benchmark of the relaxed online long convolution on one MI355X.

One "step" is one whole online generation: reset, then L positions of
lcsm_step for all M layers (red cells and batched gray tiles of Alg. 3), with
teacher-forced inputs already resident in HBM (a ring of pre-generated input
slabs).  The metric is mixer tokens/s = B * L / (seconds per step).

With --graph (default) the L per-position launches of one generation are
captured once into a HIP graph and the graph is replayed per step (the
per-token dispatch of the paper's CUDA-graph variant); --no-graph issues
every launch from the host.

Printed: one JSON line, with
  roofline      the kernel with the largest share of GPU time: its algorithmic
                bytes per launch over its average launch duration, measured
                with HIP events on the library's stream in a per-launch pass
                (event overhead measured with empty event pairs and
                subtracted);
  cpu_baseline  the CPU oracle (relaxed tiling, fp64 numpy, as it stands) on
                a bounded sample of columns of the same workload, spread over
                worker processes;
  closed_loop   the same generation with the workload's own feedback (the
                built-in tanh chain, lcsm_step_chain) instead of
                teacher-forced inputs, dispatched the same way;
  prefill       a prompt through lcsm_prefill against the same positions
                stepped;
  half_state    the timed generations again with half-state storage (T of
                the L state rows per layer), and the bytes it saves;
  data_dependent  generations with data-dependent filters (rho_t revealed
                with y_t, the parallelogram tiles of Alg. 5);
  synthetic_model  generations of the synthetic end-to-end model (per layer
                the mixer and an MLP block of hidden 2D with GELU, the next
                token = last layer's output + noise), with the mixer's share.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# The largest single-GPU workload (1M columns, 68.7 GB of state, 1.77 TB of
# algorithmic traffic per generation).
DEFAULT_WORKLOAD = "m32b16d2048l16k"
RING = 256  # input slabs kept resident
# A generation is replayed as a chain of HIP graphs, none larger than a
# bounded number of kernel nodes: a single graph of about 131k nodes (one
# generation of 131072 positions) and one of about 1.08M nodes (16384
# positions of the 32-layer synthetic model, 66 launches each) crashed the
# process while it was recorded or instantiated; graphs of up to about 33k
# nodes are known good.  Positions per graph of the library's recorder
# (lcsm_graph_capture: one or two launches per position, a few hundred at
# the rare largest tiles), and the node budget of the bench's own chains.
GRAPH_SEG = 8192
GRAPH_MAX_NODES = 16384


def parse():
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=5)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--workload", default=DEFAULT_WORKLOAD)
    p.add_argument("--graph", dest="graph", action="store_true", default=True)
    p.add_argument("--no-graph", dest="graph", action="store_false")
    p.add_argument("--graph-seg", type=int, default=GRAPH_SEG,
                   help="positions per HIP graph of a replayed generation")
    p.add_argument("--direct-max-u", type=int, default=0, help="0 = library default")
    p.add_argument("--lds-fft-max-n", type=int, default=0, help="0 = library default")
    p.add_argument("--scratch-mib", type=int, default=0, help="0 = library default")
    p.add_argument("--col-tile-form", type=int, default=0,
                   help="1: column tiles on transposed chunks instead of the column-major mirror")
    p.add_argument("--col-fft-min-n", type=int, default=0,
                   help="smallest 2U of the column-chunk FFT tiles (0 = library default, "
                        "above 16384 = off)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-budget", type=float, default=20.0, help="seconds of oracle work, about")
    p.add_argument("--no-kernel-pass", action="store_true")
    p.add_argument("--no-prefill", dest="prefill", action="store_false", default=True,
                   help="skip timing the prompt prefill against the same positions stepped online")
    p.add_argument("--no-dd", dest="dd", action="store_false", default=True,
                   help="skip the generations with data-dependent filters")
    p.add_argument("--no-synth", dest="synth", action="store_false", default=True,
                   help="skip the synthetic end-to-end model (MLP blocks + noise sampler)")
    p.add_argument("--no-half-state", dest="half_state", action="store_false", default=True,
                   help="skip the generations with half-state storage")
    p.add_argument("--extra-steps", type=int, default=1,
                   help="timed generations of each extra leg (closed loop, half-state, "
                        "data-dependent, synthetic model)")
    p.add_argument("--extra-warmup", type=int, default=1, help="untimed generations of each extra leg")
    p.add_argument("--synth-max-bytes", type=float, default=8e12,
                   help="the synthetic model is timed over the first positions whose MLP weight "
                        "reads stay below this many bytes (all L when they do)")
    p.add_argument("--baselines", default="",
                   help="comma-separated lazy/eager baselines to time over whole generations "
                        "(lazy, lazy_np, eager, eager_np; 'all' for the four), reported as the "
                        "paper's speed-up over parallel Lazy")
    p.add_argument("--baseline-warmup", type=int, default=0,
                   help="untimed baseline generations before the timed one")
    p.add_argument("--no-closed-loop", dest="closed_loop", action="store_false", default=True,
                   help="skip timing the closed-loop generation (the built-in tanh chain feeding each "
                        "layer's output into the next input)")
    p.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                   help="only run a plain elementwise copy of MIB MiB 5 times (counter calibration)")
    p.add_argument("--traffic-from", metavar="DIR", default=None,
                   help="only convert rocprofv3 FETCH_SIZE/WRITE_SIZE runs under DIR (pmc_copy_*, "
                        "pmc_bench_*) into profiles/traffic.json and a text summary")
    p.add_argument("--trace-from", metavar="DIR", default=None,
                   help="only summarise a rocprofv3 kernel trace under DIR per (kernel, U), "
                        "grouped as the per-launch pass groups launches")
    p.add_argument("--bracket", default="",
                   help="with --trace-from: comma-separated bench JSON outputs of the same command "
                        "without the profiler (before and after), quoted beside the trace")
    p.add_argument("--counters-from", metavar="DIR", default=None,
                   help="only summarise rocprofv3 --pmc runs, one derived counter per DIR/<name>, "
                        "per kernel into profiles/counters_<workload>.txt")
    p.add_argument("--sweep-from", metavar="DIR", default=None,
                   help="only tabulate bench JSON outputs DIR/sweep_<label>.json (one tile-kind "
                        "option set each) per tile size into profiles/crossover_<workload>.txt")
    p.add_argument("--command", default="", help="command line quoted in a written summary")
    p.add_argument("--copy-mib", type=int, default=1024, help="size the copy probe ran with")
    p.add_argument("--copy-scalar", action="store_true",
                   help="copy probe with 4-byte accesses per lane (a one-element offset keeps torch "
                        "from vectorising) instead of 16-byte vector accesses")
    p.add_argument("--closed-loop-once", action="store_true",
                   help="one graph-replayed closed-loop generation with progress lines (the dispatches a "
                        "kernel trace of the closed loop should see); no timing and no metric")
    p.add_argument("--trace-name", default="kernels",
                   help="--trace-from writes profiles/<name>_<workload>.txt")
    p.add_argument("--positions", type=int, default=0, metavar="P",
                   help="only run the first P positions of one generation from the host, printing "
                        "progress (for counter runs: few dispatches); prints no metric")
    return p.parse_args()


# ----------------------------------------------------------------- algorithmic bytes
def launch_bytes(name, U, w):
    """Algorithmic HBM bytes of one position's launch(es) for all M layers.

    Per column (m, b, d): the red cell reads y_t and acc_t and writes z_t and
    the slot (16 B); a gray tile of side U reads the U inputs (4(U-1) more:
    y_t is the red cell's) and reads and writes the U destination
    accumulators (8U).  Per (m, d): the lags 1..2U-1 of a direct tile
    (4(2U-1)) or the U+1 complex bins of the cached spectrum of an FFT tile
    (8(U+1)).  "fused": red cell + direct tile (U = 0: red cell only);
    "fft_lds"/"fft_hbm": red cell + FFT tile."""
    cols = w.M * w.B * w.D
    md = w.M * w.D
    if U == 0:
        return 16 * cols
    tile_cols = (16 + 4 * (U - 1) + 8 * U) * cols
    if name == "fused":
        return tile_cols + 4 * (2 * U - 1) * md
    return tile_cols + 8 * (U + 1) * md


def generation_bytes(w):
    """Algorithmic HBM bytes of one whole generation of the fixed-filter path
    (teacher-forced, or the closed loop, whose chain reads x_t in place of
    y_t): per position the red cell (16 B per column) and the gray tile of
    i = t+1 as launch_bytes counts it, with the library's default kind per U
    (direct lags up to U = 32, and U = 64 below 2^14 columns; cached spectra
    above) and the destination clipped at L."""
    cols = w.M * w.B * w.D
    md = w.M * w.D
    dmax = 64 if cols < (1 << 14) else 32
    total = 0
    for t in range(w.L):
        total += 16 * cols
        i = t + 1
        if i >= w.L:
            continue
        U = i & -i
        total += (4 * (U - 1) + 8 * min(U, w.L - i)) * cols
        total += (4 * (2 * U - 1) if U <= dmax else 8 * (U + 1)) * md
    return total


def dd_generation_bytes(w):
    """Algorithmic HBM bytes of one generation with data-dependent filters
    (Alg. 5, every power of two U dividing t+1): per position the red cell
    reads y_t, rho_t and acc_t, writes z_t and stores y_t and rho_t (24 B per
    column); a tile with 2U < t+1 reads its four blocks y[U,2U), rho[t-U+1, t],
    rho[U,2U) and y[t-U+1, t] (16U B), the square one of t+1 = 2U its two
    (8U B), and each reads and writes its destination rows acc[t+1, t+2U)
    clipped at L (8 B per row)."""
    cols = w.M * w.B * w.D
    total = 0
    for t in range(w.L):
        total += 24 * cols
        n = t + 1
        U = 1
        while 2 * U <= n:
            if n % U == 0:
                rows = min(t + 2 * U, w.L) - n
                if rows > 0:
                    total += ((16 if 2 * U < n else 8) * U + 8 * rows) * cols
            U *= 2
    return total


def generation_roofline(nbytes, ms):
    """A whole generation's algorithmic bytes against its measured time."""
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"algorithmic_GB": round(nbytes / 1e9, 3), "GB_s": round(gbs, 1),
            "frac_of_8TB_s": round(gbs / HBM_PEAK_GBS, 4)}


# Sources of the kernels a counter run of the timed region executes, and of
# their dispatch (the data-dependent, synthetic-model and column-chunk
# kernels never run there).
COUNTED_SOURCES = ("lcsm_api.hip", "lcsm_direct.hip", "lcsm_fft.hip", "lcsm_fft_col.hip",
                   "lcsm_fft_core.h", "lcsm_internal.h")


def source_digest():
    """Digest of the counted kernels' sources: counter profiles are valid only for it."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2410_12982_amd", "csrc")
    for f in COUNTED_SOURCES:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


def committed_traffic(kernel, U, w):
    """HBM bytes per launch from the committed counter profile, if it was
    taken on the current kernel sources and this workload; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    if data.get("source_digest") != source_digest():
        return None
    entry = data.get("kernels", {}).get(f"{w.name}:{kernel}:U={U}")
    return None if entry is None else entry.get("bytes_per_launch")


def kernel_key(name):
    """(kernel, U) of a library kernel name as the per-launch pass names it,
    or None for other kernels."""
    import re
    m = re.search(r"k_step_fused<(\d+), (true|false)>", name)
    if m:
        u = int(m.group(1))
        if m.group(2) == "false":
            return ("direct", u)
        return ("fused", u) if u else ("red", 0)
    m = re.search(r"k_fft_tile<(\d+), (true|false)(, (true|false))*(, \d+)?>", name)
    if m:
        return ("fft_lds", int(m.group(1)) // 2)
    # the column-chunk tile: two transposes around the transform, per chunk
    m = re.search(r"k_fft_coltile<(\d+)>", name)
    if m:
        return ("fft_col", int(m.group(1)) // 2)
    # the 2U = 2 NS tile as its even and odd halves: U = NS
    m = re.search(r"k_fft_coltile2<(\d+), \d+>", name)
    if m:
        return ("fft_col", int(m.group(1)))
    if "k_rows_to_cols" in name or "k_cols_to_rows" in name:
        return ("fft_col", None)
    # tiles on the column-major mirror, and the mirror's copies around them
    m = re.search(r"k_cm_tile<(\d+)>", name)
    if m:
        return ("fft_cm", int(m.group(1)) // 2)
    m = re.search(r"k_cm_tile2<(\d+), \d+>", name)
    if m:
        return ("fft_cm", int(m.group(1)))
    if "k_cm_yin" in name or "k_cm_merge" in name:
        return ("fft_cm", None)
    # the three-pass tile: rows of N2 points, columns of N1 (2U = N1 N2)
    m = re.search(r"k_fft_rows_(?:fwd|inv)<(\d+), (?:true|false)>", name)
    if m:
        return ("fft_hbm", ("N2", int(m.group(1))))
    m = re.search(r"k_fft_mid_tile<(\d+)>", name)
    if m:
        return ("fft_hbm", ("N1", int(m.group(1))))
    return None


def group_tiles(rows, value, order_key="Dispatch_Id"):
    """Per (kernel, U) key, one summed value per launch of the per-launch
    pass, from profiler rows in dispatch order.  A tile made of several
    dispatches -- a column tile (transposes and transform per chunk), a
    mirrored tile (the mirror's copies and the transform) or a three-pass
    tile (rows, columns, rows per chunk) -- is one launch together with the
    red cell dispatched before it: their values are summed into one entry,
    under the kind of its transform (the three-pass U from its row and
    column lengths).  value(row) gives a row's number."""
    import collections
    per = collections.defaultdict(list)
    rows = sorted(rows, key=lambda r: int(r[order_key]))
    multi = ("fft_col", "fft_cm", "fft_hbm")
    tile, red = None, None  # open multi-dispatch tile; last red-cell dispatch's value

    def close(t):
        if t["kind"] == "fft_hbm" and t["N1"] and t["N2"]:
            t["U"] = t["N1"] * t["N2"] // 2
        per[(t["kind"], t["U"])].append(t["v"])

    for r in rows:
        key = kernel_key(r["Kernel_Name"])
        v = value(r)
        if key and key[0] in multi:
            if tile is None:
                tile = {"kind": key[0], "U": None, "N1": 0, "N2": 0, "v": red or 0.0}
                red = None
            tile["v"] += v
            if key[0] == "fft_hbm" or (key[1] is not None and tile["kind"] != "fft_hbm"):
                tile["kind"] = key[0]  # the transform names the launch's kind
            if isinstance(key[1], tuple):
                tile[key[1][0]] = key[1][1]
            elif key[1] is not None:
                tile["U"] = key[1]
            continue
        if tile is not None:
            close(tile)
            tile = None
        if red is not None:
            per[("red", 0)].append(red)
            red = None
        if key == ("red", 0):
            red = v
        elif key:
            per[key].append(v)
    if tile is not None:
        close(tile)
    if red is not None:
        per[("red", 0)].append(red)
    return per


def tile_bytes(rows_c):
    """Counter bytes per (kernel, U) key and launch from one counter's rows."""
    return group_tiles(rows_c, lambda r: 1024.0 * float(r["Counter_Value"]))


def short_name(name):
    """Kernel name without namespaces and argument list."""
    import re
    name = re.sub(r"^void ", "", name).replace("(anonymous namespace)::", "").replace("lcsm::", "")
    return re.sub(r"\(.*$", "", name)


def trace_summary(args):
    """Per (kernel, U) launch durations from a rocprofv3 kernel trace
    (<dir>/run_kernel_trace.csv) of a bench command: the same grouping as the
    per-launch pass (a column tile = its red cell + every chunk's dispatches;
    a mirrored tile = its red cell, the mirror copies and the transform),
    with algorithmic GB/s and the fraction of 8 TB/s; then the kernels with
    the most time.  Written to profiles/<trace name>_<workload>.txt."""
    import collections
    import csv
    import glob

    import datagen
    w = datagen.WORKLOADS[args.workload]
    path = glob.glob(os.path.join(args.trace_from, "**", "*kernel_trace.csv"), recursive=True)[0]
    with open(path) as f:
        rows = list(csv.DictReader(f))
    per = group_tiles(rows, lambda r: (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3,
                      order_key="Start_Timestamp")
    lines = [f"# workload {w.name} (M={w.M} B={w.B} D={w.D} L={w.L}), library defaults",
             "# rocprofv3 kernel trace; command (from a scratch directory, TMPDIR=/tmp):",
             f"#   rocprofv3 --kernel-trace --stats --output-format csv -d <dir> -o run -- {args.command}",
             f"#   then: python3 bench.py --trace-from <dir> --workload {w.name}",
             f"# kernel sources digest {source_digest()}",
             "# Per launch as the per-launch pass groups them (durations summed over a launch's "
             "dispatches; every generation of the command, graph-replayed and per-launch):",
             "# kernel        U   launches    avg_us   total_ms  algorithmic_GB_s  frac_of_8TB_s"]
    for (name, U), v in sorted(per.items(), key=lambda kv: (kv[0][1] or 0, kv[0][0])):
        if U is None:
            continue
        name = "fused" if name == "red" else name
        avg = sum(v) / len(v)
        gbs = launch_bytes(name, U, w) / (avg * 1e-6) / 1e9
        lines.append(f"{name:12s} {U:5d} {len(v):10d} {avg:9.2f} {sum(v) / 1e3:10.2f} "
                     f"{gbs:17.1f} {gbs / HBM_PEAK_GBS:14.4f}")
    agg = collections.defaultdict(list)
    for r in rows:
        agg[short_name(r["Kernel_Name"])].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    total = sum(sum(v) for v in agg.values())
    lines.append("# Kernels by total time (torch's input generation outside the timed region included):")
    lines.append("#   calls     total_ms     avg_us    pct  kernel")
    for k, v in sorted(agg.items(), key=lambda kv: -sum(kv[1]))[:30]:
        lines.append(f"{len(v):9d} {sum(v) / 1e3:12.2f} {sum(v) / len(v):10.2f} "
                     f"{100 * sum(v) / total:6.2f}  {k}")
    blk = [d for k, v in agg.items() if k.split("<")[0] == "k_chain_block" for d in v]
    if blk:
        lines.append(f"# chained-step block launches (the closed loop's positions inside blocks of 32): "
                     f"{len(blk)} launches, {sum(blk) / len(blk):.2f} us each on average; with one "
                     f"generation in the command, {w.L / len(blk):.2f} positions per launch and "
                     f"{sum(blk) / w.L:.3f} us of block launch per position")
    for b in (x for x in args.bracket.split(",") if x):
        with open(b) as f:
            d = json.loads(f.read().strip().splitlines()[-1])
        lines.append(f"# bench line of the same command without the profiler ({os.path.basename(b)}): "
                     f"{d['ms_per_step']} ms per generation; per-launch pass (HIP events):")
        for key, v in d.get("per_level_us", {}).items():
            if not key.startswith("fused") or key in ("fused:U=1", "fused:U=32"):
                lines.append(f"#   {key:18s} {v['avg_us']:10.2f} us  {v['GB_s']} GB/s")
    prof = os.path.join(ROOT, "profiles")
    os.makedirs(prof, exist_ok=True)
    with open(os.path.join(prof, f"{args.trace_name}_{w.name}.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def counters_summary(args):
    """Mean of each derived counter per kernel over its dispatches, from
    rocprofv3 --pmc runs with one derived counter each (DIR/<counter>/...),
    written to profiles/counters_<workload>.txt."""
    import collections
    import csv
    import glob

    import datagen
    w = datagen.WORKLOADS[args.workload]
    res = collections.defaultdict(dict)
    names = []
    for sub in sorted(os.listdir(args.counters_from)):
        f = glob.glob(os.path.join(args.counters_from, sub, "**", "*counter_collection.csv"),
                      recursive=True)
        if not f:
            continue
        names.append(sub)
        acc = collections.defaultdict(list)
        with open(f[0]) as fh:
            for r in csv.DictReader(fh):
                acc[short_name(r["Kernel_Name"])].append(float(r["Counter_Value"]))
        for k, v in acc.items():
            res[k][sub] = (sum(v) / len(v), len(v))
    lines = [f"# workload {w.name} (M={w.M} B={w.B} D={w.D} L={w.L}), library defaults",
             "# rocprofv3 derived counters, one per run (mean over each kernel's dispatches):",
             f"#   rocprofv3 --pmc <counter> --output-format csv -d <dir>/<counter> -o run -- {args.command}",
             f"#   for <counter> in {' '.join(names)}; then: python3 bench.py --counters-from <dir> "
             f"--workload {w.name}",
             f"# kernel sources digest {source_digest()}",
             "# VALUBusy: percent of the time the vector ALUs issue; VALUUtilization: active lanes "
             "per VALU instruction; MfmaUtil: percent of the time the matrix cores are busy;",
             "# OccupancyPercent: resident waves against the maximum; LdsUtil, LDSBankConflict: "
             "LDS busy and bank-conflict cycles, percent.",
             f"{'kernel':46s}" + "".join(f"{n[:16]:>17s}" for n in names) + "  dispatches"]
    for k in sorted(res):
        if "at::" in k or "elementwise" in k:
            continue
        n = max(x[1] for x in res[k].values())
        lines.append(f"{k[:46]:46s}" + "".join(
            f"{res[k][c][0]:17.1f}" if c in res[k] else f"{'-':>17s}" for c in names) + f"  {n:10d}")
    prof = os.path.join(ROOT, "profiles")
    os.makedirs(prof, exist_ok=True)
    with open(os.path.join(prof, f"counters_{w.name}.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")
    # the same means as JSON, keyed by workload and stamped with the digest;
    # entries of other workloads taken on the same sources are kept
    path = os.path.join(prof, "counters.json")
    try:
        with open(path) as f:
            data = json.load(f)
    except (OSError, ValueError):
        data = {}
    if data.get("source_digest") != source_digest():
        data = {"source_digest": source_digest(), "workloads": {}}
    data["workloads"][w.name] = {
        k: dict({c: round(v[0], 2) for c, v in res[k].items()},
                dispatches=max(x[1] for x in res[k].values()))
        for k in sorted(res) if "at::" not in k and "elementwise" not in k}
    with open(path, "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
    print("\n".join(lines))


def group_kernels(kind, U):
    """Predicate on short kernel names: the dispatches one launch of (kind, U)
    is made of, as the per-launch pass groups them."""
    n = 2 * U
    if kind in ("fused", "red"):
        return lambda k: k == f"k_step_fused<{U}, true>"
    if kind == "direct":
        return lambda k: k.startswith("k_direct_tile")
    if kind == "fft_lds":
        return lambda k: k.startswith(f"k_fft_tile<{n},")
    if kind == "fft_cm":
        tile = "k_cm_tile2<" if n == 32768 else f"k_cm_tile<{n}>"
        return lambda k: k.startswith(tile) or k.startswith(("k_cm_yin", "k_cm_merge"))
    if kind == "fft_col":
        tile = "k_fft_coltile2" if n == 32768 else f"k_fft_coltile<{n}>"
        return lambda k: k.startswith((tile, "k_rows_to_cols", "k_cols_to_rows"))
    if kind == "fft_hbm":
        return lambda k: k.startswith(("k_fft_rows_fwd", "k_fft_mid_tile", "k_fft_rows_inv"))
    return lambda k: False


def committed_counters(kernel, U, w):
    """Derived-counter means of the dispatches of one (kernel, U) launch from
    the committed counter profile, if it was taken on the current kernel
    sources and this workload; else None."""
    try:
        with open(os.path.join(ROOT, "profiles", "counters.json")) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    if data.get("source_digest") != source_digest():
        return None
    table = data.get("workloads", {}).get(w.name)
    if not table:
        return None
    keep = group_kernels(kernel, U)
    got = {k: v for k, v in table.items() if keep(k)}
    return {"source": f"profiles/counters_{w.name}.txt", "kernels": got} if got else None


def limiter_of(counters, valu_busy=60.0):
    """Per kernel of a launch's committed counters: "vector ALU" where the
    vector ALUs issue at least valu_busy percent of the time, else "memory"
    (the matrix cores are idle in every mixer kernel)."""
    if not counters:
        return None
    return {k: ("vector ALU" if v.get("VALUBusy", 0.0) >= valu_busy else "memory")
            + f" (VALUBusy {v.get('VALUBusy', 0.0):.1f} %)"
            for k, v in counters["kernels"].items()}


def sweep_summary(args):
    """Per tile size, the per-launch time and algorithmic GB/s of every tile
    kind a sweep measured: DIR/sweep_<label>.json are bench outputs, each
    with one tile-kind option set (its per-launch pass times every tile size
    with the kind the options select).  Written to
    profiles/crossover_<workload>.txt."""
    import collections
    import glob

    import datagen
    w = datagen.WORKLOADS[args.workload]
    table = collections.defaultdict(dict)
    labels = []
    for path in sorted(glob.glob(os.path.join(args.sweep_from, f"sweep_{w.name}_*.json"))):
        label = os.path.basename(path)[len(f"sweep_{w.name}_"):-5]
        with open(path) as f:
            d = json.loads(f.read().strip().splitlines()[-1])
        labels.append((label, d["config"]["options"], d["ms_per_step"]))
        for key, v in d.get("per_level_us", {}).items():
            kind, u = key.split(":U=")
            table[int(u)][f"{kind} ({label})"] = (v["avg_us"], v["GB_s"])
    lines = [f"# workload {w.name} (M={w.M} B={w.B} D={w.D} L={w.L}): per-launch time of each tile "
             "size (HIP events, the red cell included) under tile-kind option sets",
             f"# command per set: python3 bench.py --workload {w.name} --steps 1 --warmup 1 "
             "<options> --no-cpu-baseline --no-closed-loop --no-prefill --no-half-state --no-dd "
             "--no-synth > <dir>/sweep_<workload>_<label>.json",
             f"# then: python3 bench.py --sweep-from <dir> --workload {w.name}",
             f"# kernel sources digest {source_digest()}"]
    for label, opts, ms in labels:
        lines.append(f"#   {label:14s} options {opts}: {ms} ms per generation")
    lines.append("# U      kind (set): avg_us / algorithmic GB/s, fastest first")
    for U in sorted(table):
        cells = sorted(table[U].items(), key=lambda kv: kv[1][0])
        lines.append(f"{U:6d}  " + "   ".join(f"{k}: {a:.2f} us / {g} GB/s" for k, (a, g) in cells))
    prof = os.path.join(ROOT, "profiles")
    os.makedirs(prof, exist_ok=True)
    with open(os.path.join(prof, f"crossover_{w.name}.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def traffic_from(args):
    """Convert counter runs into profiles/traffic.json: HBM bytes per launch
    per (workload, kernel, U), each counter scaled by what it reads for the
    copy probe (which reads and writes copy_mib MiB), stamped with the digest
    of the kernel sources they were taken on."""
    import csv
    import collections

    def rows(sub):
        with open(os.path.join(args.traffic_from, sub, "run_counter_collection.csv")) as f:
            return list(csv.DictReader(f))

    known = args.copy_mib * (1 << 20)
    scale = {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        vals = [1024.0 * float(r["Counter_Value"]) for r in rows(f"pmc_copy_{c}") if "neg" in r["Kernel_Name"]]
        scale[c] = known / (sum(vals) / len(vals))
    per = collections.defaultdict(lambda: {"FETCH_SIZE": [], "WRITE_SIZE": []})
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        for key, vals in tile_bytes(rows(f"pmc_bench_{c}")).items():
            per[key][c].extend(v * scale[c] for v in vals)
    # entries of other workloads taken on the same sources are kept
    path = os.path.join(ROOT, "profiles", "traffic.json")
    kept = {}
    try:
        with open(path) as f:
            old = json.load(f)
        if old.get("source_digest") == source_digest():
            kept = {k: v for k, v in old.get("kernels", {}).items()
                    if not k.startswith(args.workload + ":")}
    except (OSError, ValueError):
        pass
    kernels = {}
    for (name, U), v in sorted(per.items(), key=lambda kv: (kv[0][1] or 0, kv[0][0])):
        if U is None or not v["FETCH_SIZE"] or not v["WRITE_SIZE"]:
            continue
        fb = sum(v["FETCH_SIZE"]) / len(v["FETCH_SIZE"])
        wb = sum(v["WRITE_SIZE"]) / len(v["WRITE_SIZE"])
        kernels[f"{args.workload}:{name}:U={U}"] = {"bytes_per_launch": round(fb + wb),
                                                    "read_bytes": round(fb), "write_bytes": round(wb),
                                                    "dispatches": len(v["FETCH_SIZE"])}
    workloads = sorted({k.split(":")[0] for k in kept} | {args.workload})
    out = {"source_digest": source_digest(), "workloads": workloads,
           "fetch_scale": round(scale["FETCH_SIZE"], 4), "write_scale": round(scale["WRITE_SIZE"], 4),
           "commands": ["cd /tmp && export TMPDIR=/tmp && rocprofv3 --pmc {C} --output-format csv "
                        "-d <dir>/pmc_copy_{C} -o run -- python3 bench.py --copy-probe 1024",
                        "cd /tmp && export TMPDIR=/tmp && rocprofv3 --pmc {C} --output-format csv "
                        f"-d <dir>/pmc_bench_{{C}} -o run -- python3 bench.py --workload {args.workload} "
                        f"--positions {args.positions or '<P>'}",
                        "  for C in FETCH_SIZE, WRITE_SIZE; then: python3 bench.py --traffic-from <dir> "
                        f"--workload {args.workload}"],
           "kernels": dict(sorted({**kept, **kernels}.items()))}
    prof = os.path.join(ROOT, "profiles")
    os.makedirs(prof, exist_ok=True)
    with open(os.path.join(prof, "traffic.json"), "w") as f:
        json.dump(out, f, indent=1)
    import datagen
    w = datagen.WORKLOADS[args.workload]
    lines = [f"# HBM traffic per launch, workload {args.workload} (M={w.M} B={w.B} D={w.D} L={w.L})",
             "# rocprofv3 FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each scaled by what it reads "
             f"for a plain copy kernel of {args.copy_mib} MiB read + written "
             f"(FETCH_SIZE x {scale['FETCH_SIZE']:.4f}, WRITE_SIZE x {scale['WRITE_SIZE']:.4f})",
             *("# " + c for c in out["commands"]),
             f"# kernel sources digest {out['source_digest']}",
             "# kernel        U   dispatches   read_MB  write_MB  algorithmic_MB"]
    for key, v in kernels.items():
        _, name, u = key.split(":")
        U = int(u[2:])
        lines.append(f"{name:12s} {U:5d} {v['dispatches']:10d} {v['read_bytes'] / 1e6:9.3f} "
                     f"{v['write_bytes'] / 1e6:9.3f} {launch_bytes(name, U, w) / 1e6:12.3f}")
    with open(os.path.join(prof, f"traffic_{args.workload}.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    args = parse()
    if args.traffic_from:
        traffic_from(args)
        return
    if args.trace_from:
        trace_summary(args)
        return
    if args.counters_from:
        counters_summary(args)
        return
    if args.sweep_from:
        sweep_summary(args)
        return
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(this build has no multi-GPU path).", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_probe:
        copy_probe(args.copy_probe, torch, args.copy_scalar)
        return

    import datagen
    import paper_2410_12982_amd.lcsm as lcsm

    w = datagen.WORKLOADS[args.workload]
    if args.positions:
        counter_run(args, w, torch, datagen, lcsm)
        return
    if args.closed_loop_once:
        closed_loop_once(args, w, torch, datagen, lcsm)
        return
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    opts = {k: v for k, v in (("direct_max_u", args.direct_max_u),
                              ("lds_fft_max_n", args.lds_fft_max_n),
                              ("scratch_mib", args.scratch_mib),
                              ("col_fft_min_n", args.col_fft_min_n),
                              ("col_tile_form", args.col_tile_form)) if v} or None

    print(f"# workload {w.name}: M={w.M} B={w.B} D={w.D} L={w.L} graph={args.graph}",
          file=sys.stderr, flush=True)
    filters = datagen.filters_torch(w, dev)
    R = min(RING, w.L)
    y = datagen.y_torch(w, dev, 0, R)                 # [R, M, B, D] resident in HBM
    z = torch.empty_like(y)
    ms = timed_generations(w, filters, y, z, opts, lcsm, torch, dev, args, verbose=True)
    value = w.B * w.L / (ms / 1e3)
    torch.cuda.synchronize()

    roofline, levels = None, {}
    if not args.no_kernel_pass:
        roofline, levels = kernel_pass(w, filters, y, z, opts, lcsm, torch)
        # the per-launch floor this launch-bound path sits on, measured live
        floor_us = launch_floor(w, torch, dev)
        roofline["launch_floor"] = {
            "us_per_launch": round(floor_us, 3),
            "how": "graph-replayed elementwise kernels on a tensor of one position's M*B*D floats",
            "generation_us_per_position": round(1e3 * ms / w.L, 3)}
        # a kernel whose launches last about as long as an almost empty
        # graph-replayed launch is bound by the launch, not by HBM
        if roofline["avg_launch_us"] < 2.0 * floor_us:
            roofline["bound"] = "launch"
        # what the hardware counters say about those dispatches (vector-ALU
        # and matrix-core busy, occupancy), when taken on these sources
        kname, kU = roofline["kernel"].split(" U=")
        roofline["counters"] = committed_counters(kname, int(kU), w)
        roofline["limiter"] = limiter_of(roofline["counters"])

    def release():
        # each leg's contexts hold tens of GB; give torch's cached blocks back
        # so that the next leg's library-allocated workspace fits
        import gc
        gc.collect()
        torch.cuda.synchronize()
        torch.cuda.empty_cache()

    release()
    closed = None
    if args.closed_loop:
        closed = closed_loop(w, filters, opts, lcsm, torch, dev, args)
        release()

    prefill = None
    if args.prefill:
        prefill = prefill_timing(w, filters, opts, lcsm, torch, dev)
        release()

    half = None
    if args.half_state:
        half = half_state_timing(w, filters, y, z, opts, ms, lcsm, torch, dev, args)
        release()

    dd = None
    if args.dd:
        dd = dd_timing(w, ms, lcsm, torch, dev, args)
        release()

    synth = None
    if args.synth:
        synth = synth_timing(w, filters, opts, ms, lcsm, torch, dev, args)
        release()

    base = None
    if args.baselines:
        kinds = (["lazy", "lazy_np", "eager", "eager_np"] if args.baselines == "all"
                 else [k for k in args.baselines.split(",") if k])
        base = baselines_timing(w, filters, y, ms, kinds, lcsm, torch, dev, args, synth)
        release()

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
                   "options": opts or "default", "graph": args.graph,
                   "parallelism": "single-gpu"},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    # every generation-shaped leg against its algorithmic bytes
    gen = generation_bytes(w)
    out["generation"] = generation_roofline(gen, ms)
    if closed:
        closed["generation"] = generation_roofline(gen, closed["ms_per_step"])
    if half:
        half["generation"] = generation_roofline(gen, half["ms_per_step"])
    if dd:
        dd["generation"] = generation_roofline(dd_generation_bytes(w), dd["ms_per_step"])
    if levels:
        out["per_level_us"] = levels
    if closed:
        out["closed_loop"] = closed
    if prefill:
        out["prefill"] = prefill
    if half:
        out["half_state"] = half
    if synth:
        out["synthetic_model"] = synth
    if dd:
        out["data_dependent"] = dd
    if base:
        out["baselines"] = base
    print(json.dumps(out), flush=True)


def counter_run(args, w, torch, datagen, lcsm):
    """The first P positions of one generation, launched from the host (the
    dispatches a counter run should see), with a progress line after every
    set-up phase and every 256 positions.  No timing and no metric.  Under a
    counter profiler every dispatch is serialised, so the set-up keeps its
    dispatch count small: filters generated 8 layers per pass (a few hundred
    elementwise kernels instead of a few thousand) and a ring of 16 input
    slabs (the counted kernels' traffic does not depend on the values)."""
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    opts = {k: v for k, v in (("direct_max_u", args.direct_max_u),
                              ("lds_fft_max_n", args.lds_fft_max_n),
                              ("scratch_mib", args.scratch_mib),
                              ("col_fft_min_n", args.col_fft_min_n),
                              ("col_tile_form", args.col_tile_form)) if v} or None
    P = min(args.positions, w.L)

    def say(msg):
        print(f"# {msg}", file=sys.stderr, flush=True)

    say(f"counter run {w.name}: {P} positions")
    filters = datagen.filters_torch(w, dev, m_chunk=8)
    torch.cuda.synchronize()
    say("filters generated")
    R = min(16, w.L)
    y = datagen.y_torch(w, dev, 0, R)
    z = torch.empty_like(y)
    torch.cuda.synchronize()
    say(f"input ring of {R} slabs generated")
    ctx = lcsm.Lcsm(filters, w.B, options=opts)
    torch.cuda.synchronize()
    say("context initialised (filter re-layout, state cleared, spectra of every FFT tile size)")
    del filters
    for t in range(P):
        ctx.step(y[t % R], z[t % R])
        if (t + 1) % 256 == 0 or t + 1 == P:
            torch.cuda.synchronize()
            say(f"position {t + 1} of {P}")
    ctx.close()
    print(json.dumps({"counter_run": True, "workload": w.name, "positions": P}), flush=True)


def closed_loop_once(args, w, torch, datagen, lcsm):
    """One closed-loop generation as the closed-loop leg dispatches it
    (recorded by the library as a chain of HIP graphs, then replayed once),
    with a progress line after every phase.  No timing and no metric."""
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    def say(msg):
        print(f"# {msg}", file=sys.stderr, flush=True)

    say(f"closed-loop generation {w.name}")
    filters = datagen.filters_torch(w, dev)
    R = min(RING, w.L)
    x = datagen.x_torch(w, dev, 0, R)
    z = torch.empty_like(x)
    stream = torch.cuda.Stream(dev)
    torch.cuda.synchronize()
    say("filters and input ring generated")
    ctx = lcsm.Lcsm(filters, w.B, stream=stream)
    torch.cuda.synchronize()
    say("context initialised")
    del filters
    graph = ctx.capture(x, z, n=w.L, chain=True, seg=args.graph_seg)
    say(f"generation recorded ({graph.segments} graphs)")
    graph.launch()
    torch.cuda.synchronize()
    say("generation replayed")
    graph.close()
    ctx.close()
    print(json.dumps({"closed_loop_once": True, "workload": w.name, "positions": w.L}), flush=True)


def copy_probe(mib, torch, scalar=False):
    """A plain elementwise kernel reading and writing mib MiB each (b = -a),
    five times: the reference for scaling the HBM byte counters.  scalar: the
    views start one element into their buffers, so torch cannot use vector
    accesses and every lane moves 4 bytes."""
    n = mib * (1 << 20) // 4
    a = torch.ones(n + 1, dtype=torch.float32, device="cuda:0")
    b = torch.empty_like(a)
    src, dst = (a[1:], b[1:]) if scalar else (a[:n], b[:n])
    torch.cuda.synchronize()
    for _ in range(5):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_mib": mib, "scalar": scalar, "bytes_read": 4 * n,
                      "bytes_written": 4 * n}), flush=True)


def launch_floor(w, torch, dev, n=2048):
    """Microseconds per launch of n back-to-back elementwise kernels (x += 1
    on M*B*D floats, one position's slab) replayed from one HIP graph: the
    cost of a launch that does one read and one write per element."""
    x = torch.zeros(w.M * w.B * w.D, dtype=torch.float32, device=dev)
    s = torch.cuda.Stream(dev)
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        for _ in range(n):
            x.add_(1.0)
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    best = float("inf")
    for _ in range(3):
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1))
    del g
    return 1e3 * best / n


def kernel_pass(w, filters, y, z, opts, lcsm, torch):
    """Average duration of one position's launch(es) per tile kind and side U
    over one generation, with HIP events on the library's stream (torch's
    current stream), bracketing each lcsm_step exactly as the timed region
    issues it: one launch for the red cell fused with a direct tile (U <= 64)
    or with a single-pass FFT tile (2U <= 4096), red cell + tile launches
    otherwise.  Empty event pairs, recorded as often as bracketed ones,
    measure the event overhead, which is subtracted."""
    stream = torch.cuda.current_stream()
    ctx = lcsm.Lcsm(filters, w.B, options=opts, stream=stream)
    R = y.shape[0]
    plans = [ctx.plan(t) for t in range(w.L)]
    ctx.reset()
    torch.cuda.synchronize()
    pool = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(4)) for _ in range(2048)]
    recs, empty, k = [], [], 0
    for t in range(w.L):
        i, U, n, kind = plans[t]
        a, b, c, d = pool[k % len(pool)]
        c.record(stream)
        d.record(stream)
        a.record(stream)
        ctx.step(y[t % R], z[t % R])
        b.record(stream)
        name = {lcsm.TILE_NONE: "fused", lcsm.TILE_DIRECT: "fused"}.get(kind, lcsm.TILE_KIND_NAMES[kind])
        recs.append((name, U, a, b))
        empty.append((c, d))
        k += 1
        if k % len(pool) == 0:
            torch.cuda.synchronize()
            recs = [(r[0], r[1], r[2].elapsed_time(r[3])) if len(r) == 4 else r for r in recs]
            empty = [e if isinstance(e, float) else e[0].elapsed_time(e[1]) for e in empty]
    torch.cuda.synchronize()
    recs = [(r[0], r[1], r[2].elapsed_time(r[3])) if len(r) == 4 else r for r in recs]
    empty = [e if isinstance(e, float) else e[0].elapsed_time(e[1]) for e in empty]
    ctx.close()
    overhead_ms = sorted(empty)[len(empty) // 2]
    agg = {}
    for name, U, dur in recs:
        s = agg.setdefault((name, U), [0.0, 0])
        s[0] += max(dur - overhead_ms, 0.0)
        s[1] += 1
    total = sum(v[0] for v in agg.values())
    levels = {f"{name}:U={U}": {"launches": n, "avg_us": round(1e3 * tot / n, 3),
                                "total_ms": round(tot, 3),
                                "GB_s": round(launch_bytes(name, U, w) / (tot / n / 1e3) / 1e9, 1)
                                if tot > 0 else None}
              for (name, U), (tot, n) in sorted(agg.items(), key=lambda kv: kv[0][1])}
    (name, U), (tot, n) = max(agg.items(), key=lambda kv: kv[1][0])
    avg_s = tot / n / 1e3
    nbytes = launch_bytes(name, U, w)
    achieved = nbytes / avg_s / 1e9
    roofline = {"bound": "hbm", "kernel": f"{name} U={U}", "achieved": round(achieved, 2),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 5),
                "traffic": committed_traffic(name, U, w), "bytes_per_launch": nbytes,
                "avg_launch_us": round(avg_s * 1e6, 3), "launches": n,
                "event_overhead_us": round(1e3 * overhead_ms, 3),
                "share_of_gpu_time": round(tot / total, 4)}
    # the largest tile kernel, for the bandwidth of the FFT path
    big = [(key, v) for key, v in agg.items() if key[0] != "fused"]
    if big:
        (bname, bU), (btot, bn) = max(big, key=lambda kv: kv[0][1])
        bavg = btot / bn / 1e3
        bbytes = launch_bytes(bname, bU, w)
        roofline["largest_tile"] = {"kernel": f"{bname} U={bU}", "bytes_per_launch": bbytes,
                                    "avg_launch_us": round(bavg * 1e6, 3),
                                    "achieved": round(bbytes / bavg / 1e9, 2),
                                    "frac": round(bbytes / bavg / 1e9 / HBM_PEAK_GBS, 5),
                                    "traffic": committed_traffic(bname, bU, w)}
    # every FFT tile size against the 50 % HBM gate on algorithmic bytes
    roofline["fft_tiles_vs_gate"] = {
        f"{k[0]} U={k[1]}": round(launch_bytes(k[0], k[1], w) / (v[0] / v[1] / 1e3) / 1e9
                                  / HBM_PEAK_GBS, 4)
        for k, v in sorted(agg.items(), key=lambda kv: kv[0][1]) if k[0] != "fused" and v[0] > 0}
    return roofline, levels


def time_steps(one_step, torch, args, verbose=False, extra=None):
    """Untimed warm-up calls of one_step, then timed ones, bracketed by events
    on the current stream.  The timed region uses args.warmup / args.steps;
    an extra leg (extra = its name) uses args.extra_warmup / args.extra_steps
    and prints a line per generation.  Returns ms per step."""
    warmup, steps = (args.warmup, args.steps) if extra is None else (args.extra_warmup,
                                                                     args.extra_steps)
    for k in range(warmup):
        one_step()
        if extra:
            torch.cuda.synchronize()
            print(f"# {extra}: warm-up {k + 1}/{warmup}", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    if verbose:
        print(f"# warmup done ({warmup})", file=sys.stderr, flush=True)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    ev0.record()
    for _ in range(steps):
        one_step()
    ev1.record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms = ev0.elapsed_time(ev1) / steps
    if verbose or extra:
        print(f"# {extra or 'timed'}: {steps} steps, {ms:.3f} ms/step (wall "
              f"{1e3 * t_wall / steps:.3f})", file=sys.stderr, flush=True)
    return ms


class GraphChain:
    """A generation of a context without the library's own recorder (the
    data-dependent, synthetic-model and baseline contexts) as a chain of
    torch HIP graphs: issue(p0, p1) queues positions [p0, p1) (the reset with
    p0 = 0) on the capture stream, and each graph takes as many positions as
    keep it within GRAPH_MAX_NODES kernel nodes given at most per_position
    launches per position (and at most seg positions)."""

    def __init__(self, torch, stream, L, seg, issue, per_position):
        self.positions = max(1, min(seg, GRAPH_MAX_NODES // max(1, per_position)))
        self.graphs = []
        for p0 in range(0, L, self.positions):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=stream):
                issue(p0, min(L, p0 + self.positions))
            self.graphs.append(g)
        torch.cuda.synchronize()

    def replay(self):
        for g in self.graphs:
            g.replay()

    def close(self):
        self.graphs = []


def timed_generations(w, filters, y, z, opts, lcsm, torch, dev, args, verbose=False, extra=None):
    """Teacher-forced generations of all L positions (inputs from the ring y
    resident in HBM), recorded once by the library as a chain of HIP graphs
    (lcsm_graph_capture: reset + L steps, at most args.graph_seg positions per
    graph) and replayed per step, or launched from the host with --no-graph:
    warmup untimed, then args.steps timed with events.  Returns ms per
    generation."""
    R = y.shape[0]
    stream = torch.cuda.Stream(dev) if args.graph else torch.cuda.current_stream(dev)
    ctx = lcsm.Lcsm(filters, w.B, options=opts, stream=stream)
    torch.cuda.synchronize()
    graph = None
    if args.graph:
        graph = ctx.capture(y, z, n=w.L, seg=args.graph_seg)
        torch.cuda.synchronize()
        if verbose:
            print(f"# recorded: {graph.segments} graph(s) of <= {args.graph_seg} positions",
                  file=sys.stderr, flush=True)
        one_step = graph.launch
    else:
        def one_step():
            ctx.reset()
            for t0 in range(0, w.L, R):
                ctx.run(y, z, n=min(R, w.L - t0))
    with torch.cuda.stream(stream):
        ms = time_steps(one_step, torch, args, verbose, extra)
    if graph is not None:
        graph.close()
    ctx.close()
    del ctx
    torch.cuda.synchronize()
    return ms


def baselines_timing(w, filters, y, ms_relaxed, kinds, lcsm, torch, dev, args, synth=None):
    """Whole generations of the lazy and eager baselines (lcsm_base_step, the
    paper's Lazy/Eager and their per-layer *_NP variants) on the same
    teacher-forced ring inputs, each replayed as a chain of HIP graphs like
    the timed region: args.baseline_warmup untimed, then one timed
    generation (a lazy generation is O(L^2): tens of seconds at 32K
    positions).  Reports each one's time and the relaxed generation's
    speed-up over it; with the synthetic model's time, the end-to-end
    speed-up over a model whose mixer is parallel Lazy, taking the model's
    non-mixer time as unchanged."""
    R = y.shape[0]
    out = {}
    for kind in kinds:
        stream = torch.cuda.Stream(dev)
        ctx = lcsm.Base(kind, filters, w.B, stream=stream)
        z = torch.empty_like(y)
        torch.cuda.synchronize()

        def issue(p0, p1):
            if p0 == 0:
                ctx.reset()
            for t in range(p0, p1):
                ctx.step(y[t % R], z[t % R])

        print(f"# baseline {kind}: recording", file=sys.stderr, flush=True)
        # lazy: partial sums + reduction; eager: one launch; per layer with _np
        per_pos = (2 if kind.startswith("lazy") else 1) * (w.M if kind.endswith("_np") else 1)
        chain = GraphChain(torch, stream, w.L, args.graph_seg, issue, per_pos)
        with torch.cuda.stream(stream):
            for _ in range(args.baseline_warmup):
                chain.replay()
            torch.cuda.synchronize()
            # graph by graph, with a progress line after each (a lazy or eager
            # generation of 131072 positions takes minutes); the timed region
            # spans them all, the waits between graphs included
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for k, g in enumerate(chain.graphs):
                g.replay()
                torch.cuda.synchronize()
                print(f"# baseline {kind}: graph {k + 1} of {len(chain.graphs)} "
                      f"({chain.positions} positions each)", file=sys.stderr, flush=True)
            e1.record()
        torch.cuda.synchronize()
        bms = e0.elapsed_time(e1)
        chain.close()
        ctx.close()
        print(f"# baseline {kind}: {bms:.1f} ms per generation", file=sys.stderr, flush=True)
        out[kind] = {"ms_per_step": round(bms, 3), "tokens_per_s": round(w.B * w.L / (bms / 1e3), 1),
                     "relaxed_speedup": round(bms / ms_relaxed, 2)}
    if "lazy" in out:
        out["speedup_over_parallel_lazy"] = out["lazy"]["relaxed_speedup"]
        if synth and synth.get("positions") == w.L:
            lazy_model = synth["ms_per_step"] - ms_relaxed + out["lazy"]["ms_per_step"]
            out["end_to_end_speedup_over_parallel_lazy"] = {
                "value": round(lazy_model / synth["ms_per_step"], 2),
                "how": "synthetic model with the parallel-Lazy mixer estimated as the model's time "
                       "minus the relaxed mixer's plus the Lazy mixer's, over the model's time"}
    return out


def half_state_timing(w, filters, y, z, opts, ms_full, lcsm, torch, dev, args):
    """The same generations with half-state storage (App. C: T state rows per
    layer instead of L, the tile of i = T storing over its own inputs), timed
    the same way; with the state bytes of both forms."""
    hopts = dict(opts or {}, half_state=1)
    try:
        full_b = lcsm.workspace_bytes(w.M, w.B, w.D, w.L, opts)
        half_b = lcsm.workspace_bytes(w.M, w.B, w.D, w.L, hopts)
    except lcsm.LcsmError as e:  # the tile of side T is a direct tile here
        return {"skipped": str(e)}
    print("# half-state generations", file=sys.stderr, flush=True)
    ms = timed_generations(w, filters, y, z, hopts, lcsm, torch, dev, args, extra="half-state")
    T = 1
    while 2 * T < w.L:
        T *= 2
    return {"T": T, "ms_per_step": round(ms, 4), "tokens_per_s": round(w.B * w.L / (ms / 1e3), 1),
            "time_vs_full_state": round(ms / ms_full, 4),
            "state_bytes": 4 * w.M * T * w.B * w.D, "state_bytes_full": 4 * w.M * w.L * w.B * w.D,
            "workspace_bytes": half_b, "workspace_bytes_full": full_b}


def dd_timing(w, ms_fixed, lcsm, torch, dev, args):
    """Generations with data-dependent filters (lcsm_dd_step: rho_t revealed
    with y_t; every power of two U dividing t+1 gets a parallelogram tile),
    teacher-forced y and rho resident in HBM, dispatched like the timed
    region (a chain of HIP graphs).  ms_fixed: the data-independent
    generation, for the ratio."""
    import datagen
    try:
        lcsm.dd_workspace_bytes(w.M, w.B, w.D, w.L)
    except lcsm.LcsmError as e:   # a shape the context rejects
        return {"skipped": str(e)}
    R = min(RING, w.L)
    y = datagen.y_torch(w, dev, 0, R)
    rho = datagen.rho_torch(w, dev, 0, R)
    z = torch.empty_like(y)
    stream = torch.cuda.Stream(dev) if args.graph else torch.cuda.current_stream(dev)
    ctx = lcsm.Dd(w.M, w.B, w.D, w.L, stream=stream)
    torch.cuda.synchronize()

    def issue(p0, p1):
        if p0 == 0:
            ctx.reset()
        for t in range(p0, p1):
            ctx.step(y[t % R], rho[t % R], z[t % R])

    # the red cell with the small tiles, plus one launch per larger U dividing t+1
    per_pos = 1 + max(1, (w.L - 1).bit_length())
    chain = GraphChain(torch, stream, w.L, args.graph_seg, issue, per_pos) if args.graph else None
    one = chain.replay if chain else (lambda: issue(0, w.L))
    print("# data-dependent generations", file=sys.stderr, flush=True)
    with torch.cuda.stream(stream):
        dms = time_steps(one, torch, args, extra="data-dependent")
    if chain:
        chain.close()
    ctx.close()
    return {"ms_per_step": round(dms, 4), "tokens_per_s": round(w.B * w.L / (dms / 1e3), 1),
            "time_vs_fixed_filters": round(dms / ms_fixed, 3), "graph": bool(chain)}


def synth_timing(w, filters, opts, ms_mixer, lcsm, torch, dev, args):
    """Generations of the synthetic end-to-end model (lcsm_synth_step: per
    layer the mixer and an MLP block of hidden 2D with GELU; the next token
    = last layer's output + noise), dispatched like the timed region (a chain
    of HIP graphs): args.extra_warmup untimed, then args.extra_steps timed
    with events.  When a generation would read more than args.synth_max_bytes
    of MLP weights (the 1M-column workload reads 2.1 GB per position), the
    model is timed over its first P positions (P a power of two) instead.
    ms_mixer: the teacher-forced mixer generation time, for the mixer's share
    of the model's time (per position, over the whole generation)."""
    import datagen
    wbytes = 4 * w.M * (4 * w.D * w.D + 3 * w.D)
    P = w.L
    if wbytes * w.L > args.synth_max_bytes:
        P = 256
        while 2 * P < w.L and 2 * P * wbytes <= args.synth_max_bytes:
            P *= 2
    R = min(RING, w.L)
    weights = datagen.mlp_weights_torch(w, dev)
    eps = datagen.noise_torch(w, dev, 0, R)
    act = torch.empty((R, w.M, w.B, w.D), dtype=torch.float32, device=dev)
    stream = torch.cuda.Stream(dev) if args.graph else torch.cuda.current_stream(dev)
    model = lcsm.Synth(filters, *weights, w.B, options=opts, stream=stream)
    torch.cuda.synchronize()

    def issue(p0, p1):
        if p0 == 0:
            model.reset()
        for t in range(p0, p1):
            model.step(eps[t % R], act[t % R])

    # sampler/red cell, two products per layer and 16 batch rows, the gray tiles
    per_pos = 2 + 2 * w.M * (-(-w.B // 16)) + 8
    chain = GraphChain(torch, stream, P, args.graph_seg, issue, per_pos) if args.graph else None
    one = chain.replay if chain else (lambda: issue(0, P))
    print(f"# synthetic-model generations ({P} of {w.L} positions)", file=sys.stderr, flush=True)
    with torch.cuda.stream(stream):
        sms = time_steps(one, torch, args, extra="synthetic model")
    if chain:
        chain.close()
    model.close()
    us_pos = 1e3 * sms / P
    out = {"positions": P, "ms_per_step": round(sms, 4), "tokens_per_s": round(w.B * P / (sms / 1e3), 1),
           "us_per_position": round(us_pos, 3),
           "mixer_share": round(1e3 * ms_mixer / w.L / us_pos, 4),
           "weight_bytes_per_position": wbytes,
           "weight_GB_s": round(wbytes / (us_pos * 1e-6) / 1e9, 1),
           "launches_per_position": 2 * w.M + 2,
           "graph": bool(chain)}
    if P < w.L:
        out["note"] = (f"timed over the first {P} positions (whole generations would read "
                       f"{wbytes * w.L / 1e12:.1f} TB of weights)")
    return out


def closed_loop(w, filters, opts, lcsm, torch, dev, args):
    """Closed-loop generations (lcsm_step_chain: y^0_t = 0.5 tanh(z^{M-1}_{t-1})
    + x^0_t, y^m_t = 0.5 tanh(z^{m-1}_t) + x^m_t), dispatched like the timed
    region (recorded by the library as a chain of HIP graphs): warmup untimed,
    then steps timed with events."""
    import datagen
    R = min(RING, w.L)
    x = datagen.x_torch(w, dev, 0, R)
    z = torch.empty_like(x)
    stream = torch.cuda.Stream(dev) if args.graph else torch.cuda.current_stream(dev)
    ctx = lcsm.Lcsm(filters, w.B, options=opts, stream=stream)
    torch.cuda.synchronize()
    graph = ctx.capture(x, z, n=w.L, chain=True, seg=args.graph_seg) if args.graph else None

    def host_generation():
        ctx.reset()
        for t in range(w.L):
            ctx.step_chain(x[t % R], z[t % R])

    one = graph.launch if graph else host_generation
    with torch.cuda.stream(stream):
        cms = time_steps(one, torch, args, extra="closed loop")
    if graph:
        graph.close()
    ctx.close()
    return {"ms_per_step": round(cms, 4), "tokens_per_s": round(w.B * w.L / (cms / 1e3), 1),
            "graph": bool(graph)}


def prefill_timing(w, filters, opts, lcsm, torch, dev, max_bytes=2 << 30):
    """A prompt of P positions (the largest power of two with 2P <= L whose
    inputs fit in max_bytes) through lcsm_prefill against the same P
    positions through lcsm_run, each captured in a HIP graph (reset
    included) and replayed: prompt tokens/s of both."""
    import datagen
    slab = w.M * w.B * w.D * 4
    P = 1
    while 4 * P <= w.L and 2 * P * slab <= max_bytes:
        P *= 2
    y = datagen.y_torch(w, dev, 0, P)
    z = torch.empty_like(y)
    stream = torch.cuda.Stream(dev)
    ctx = lcsm.Lcsm(filters, w.B, options=opts, stream=stream)
    torch.cuda.synchronize()
    res = {}
    for mode in ("prefill", "steps"):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            ctx.reset()
            if mode == "prefill":
                ctx.prefill(y, z, P)
            else:
                ctx.run(y, z, n=P)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(3):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        res[mode] = e0.elapsed_time(e1) / 3
        del g
    ctx.close()
    return {"P": P, "ms": round(res["prefill"], 4), "steps_ms": round(res["steps"], 4),
            "prompt_tokens_per_s": round(w.B * P / (res["prefill"] / 1e3), 1),
            "speedup_vs_steps": round(res["steps"] / res["prefill"], 2)}


def _oracle_shard(arg):
    """Worker: run the relaxed-tiling oracle on a set of (b, d) columns of
    layer 0 over all L positions; returns the elapsed seconds."""
    name, b_idx, d_idx = arg
    import numpy as np

    import datagen
    from oracle import feedback
    from oracle.relaxed import relaxed_online
    w = datagen.WORKLOADS[name]
    h = datagen.filters_np(w, m_idx=[0], d_idx=d_idx)[0]          # [n_d, L]
    n = len(b_idx) * len(d_idx)
    hc = np.broadcast_to(h.T[:, None, None, :], (w.L, 1, len(b_idx), len(d_idx)))
    hc = np.ascontiguousarray(hc).reshape(w.L, 1, n)
    yc = datagen.y_np(w, m_idx=[0], b_idx=b_idx, d_idx=d_idx).reshape(w.L, 1, n)
    t0 = time.perf_counter()
    relaxed_online(hc, feedback.teacher_forced(yc))
    return time.perf_counter() - t0


def cpu_model():
    """The host CPU's model name (first 'model name' line of /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# Worker processes of the CPU baseline: the host's CPU share per GPU (a
# one-GPU machine grants 16 CPUs whatever os.cpu_count() reports).
CPU_SHARE = 16


def cpu_baseline(w, budget_s):
    """Time the CPU oracle (relaxed tiling, fp64 numpy, as it stands) on a
    bounded sample: all positions of a set of (b, d) columns, sharded over
    worker processes (one thread each); the sample grows until it takes
    about budget_s / 4 seconds of wall time or covers every column.  The rate
    is extrapolated linearly to all columns when the sample is smaller."""
    import multiprocessing as mp

    import numpy as np
    host = os.cpu_count() or 1
    workers = max(1, min(CPU_SHARE, host))
    total_cols = w.M * w.B * w.D
    env_keys = ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")
    saved = {k: os.environ.get(k) for k in env_keys}
    for k in env_keys:
        os.environ[k] = "1"
    ctx = mp.get_context("spawn")
    per = 4
    try:
        with ctx.Pool(workers) as pool:
            while True:
                nd = min(w.D, per)
                b_idx = np.arange(max(1, min(w.B, per // nd)))
                # distinct channels per worker where the workload has enough
                shards = [(w.name, b_idx, (np.arange(nd) + k * nd) % w.D) for k in range(workers)]
                # oracle time only (input generation excluded); shards run in parallel
                wall = max(pool.map(_oracle_shard, shards))
                n = len(b_idx) * nd * workers
                print(f"# cpu baseline: {n} columns in {wall:.1f} s", file=sys.stderr, flush=True)
                if wall * 4 > budget_s or n >= total_cols or per >= 4096:
                    break
                # the oracle vectorises over columns: fewer, wider shards are cheaper
                per = min(per * 4, -(-total_cols // workers))
    finally:
        for k, v in saved.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
    n = min(n, total_cols)
    value = w.B * w.L / (wall * total_cols / n)
    extrap = n < total_cols
    return {"value": round(value, 2), "unit": "tokens/s", "cores": workers, "kind": "oracle",
            "host_cpus": host, "cpu_model": cpu_model(), "extrapolated": extrap,
            "sample": f"relaxed-tiling oracle (fp64 numpy), all {w.L} positions of {n} of the "
                      f"{total_cols} columns ({workers} single-thread processes x {n // workers} "
                      f"columns of layer 0, in parallel; {workers} of the host's {host} CPUs, the "
                      f"CPU share of one GPU) in {wall:.1f} s (slowest process)"
                      + (f", extrapolated linearly to all {total_cols} columns" if extrap else "")}


if __name__ == "__main__":
    main()
