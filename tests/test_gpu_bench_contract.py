"""The benchmark's output contract, on the GPU (needs an MI355X).

bench.py runs as its own process on the smallest workload with every leg and
the CPU baseline on, and its single JSON line must carry the fields a reader
of the result relies on: the metric, the step and warm-up counts, a value
consistent with ms_per_step, the roofline object of the dominant launch (its
achieved rate equal to its bytes over its duration, its fraction equal to
achieved over peak) and the CPU baseline (the oracle, with its core count
and sample), and the whole-generation figures of the timed region and
the generation-shaped legs (their GB/s equal to the algorithmic bytes of a
generation over its time)."""
import json
import os
import subprocess
import sys

import pytest

import bench
import datagen
from gpu_harness import say

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_json_line_contract():
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "m1b1d16l1k", "--steps", "3",
           "--warmup", "1", "--cpu-budget", "2"]
    say("[bench contract] " + " ".join(cmd[1:]))
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, lines
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1
    assert d["higher_is_better"] is True and d["dtype"] == "f32"
    assert d["config"]["workload"] == "m1b1d16l1k"
    # value is B * L tokens per generation over the generation time
    B, L = d["config"]["B"], d["config"]["L"]
    assert abs(d["value"] - B * L / (d["ms_per_step"] / 1e3)) <= 1e-3 * d["value"]
    rf = d["roofline"]
    assert rf["bound"] in ("hbm", "mfma", "alu", "launch")
    assert rf["unit"] == "GB/s" and rf["peak"] == 8000.0
    achieved = rf["bytes_per_launch"] / (rf["avg_launch_us"] * 1e-6) / 1e9
    assert abs(rf["achieved"] - achieved) <= 1e-2 * achieved + 0.01
    assert abs(rf["frac"] - rf["achieved"] / rf["peak"]) <= 1e-4
    assert "traffic" in rf
    cpu = d["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["cores"] >= 1 and cpu["value"] > 0 and cpu["sample"]
    for leg in ("closed_loop", "prefill", "half_state", "data_dependent", "synthetic_model"):
        assert leg in d, leg
    # whole generations against their algorithmic bytes
    w = datagen.WORKLOADS["m1b1d16l1k"]
    for obj, nbytes in ((d, bench.generation_bytes(w)), (d["closed_loop"], bench.generation_bytes(w)),
                        (d["half_state"], bench.generation_bytes(w)),
                        (d["data_dependent"], bench.dd_generation_bytes(w))):
        g = obj["generation"]
        gbs = nbytes / (obj["ms_per_step"] * 1e-3) / 1e9
        assert abs(g["GB_s"] - gbs) <= 1e-3 * gbs + 0.1
        assert abs(g["frac_of_8TB_s"] - gbs / 8000.0) <= 1e-4
    say(f"  {d['value']:.0f} tokens/s, dominant {rf['kernel']} ({rf['bound']})")
