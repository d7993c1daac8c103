"""Host logic of bench.py (no GPU): the mapping of profiled kernel names to
the per-launch pass's (kernel, U) keys, the aggregation of counter rows into
one entry per tile, the algorithmic-bytes formula on hand-counted cases, the
digest's file list, and the refusal of more than one GPU."""
import os
import subprocess
import sys

import pytest

import bench
import datagen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("name,key", [
    ("void lcsm::(anonymous namespace)::k_step_fused<1, true>(float*, int)", ("fused", 1)),
    ("lcsm::k_step_fused<32, true>", ("fused", 32)),
    ("lcsm::k_step_fused<0, true>", ("red", 0)),
    ("lcsm::k_step_fused<8, false>", ("direct", 8)),
    ("lcsm::k_fft_tile<8192, false, true, false>", ("fft_lds", 4096)),
    ("lcsm::k_fft_tile<4096, true, true, false, 4>", ("fft_lds", 2048)),
    ("lcsm::k_fft_tile<128, true, false, false, 8>(float*, float2 const*)", ("fft_lds", 64)),
    ("lcsm::k_fft_coltile<16384>", ("fft_col", 8192)),
    ("lcsm::(anonymous namespace)::k_fft_coltile2<16384, 1>(float*, float*)", ("fft_col", 16384)),
    ("lcsm::k_fft_coltile2<16384, 0>", ("fft_col", 16384)),
    ("lcsm::k_rows_to_cols", ("fft_col", None)),
    ("lcsm::k_cols_to_rows<false>", ("fft_col", None)),
    ("void lcsm::(anonymous namespace)::k_cm_tile<2048>(float2*, unsigned long)", ("fft_cm", 1024)),
    ("lcsm::k_cm_tile2<16384, 1>", ("fft_cm", 16384)),
    ("lcsm::k_cm_yin4(float const*)", ("fft_cm", None)),
    ("lcsm::k_cm_merge4<true>", ("fft_cm", None)),
    ("lcsm::k_cm_merge<false>", ("fft_cm", None)),
    ("lcsm::k_fft_rows_fwd<4096, true>", ("fft_hbm", ("N2", 4096))),
    ("lcsm::k_fft_mid_tile<32>", ("fft_hbm", ("N1", 32))),
    ("at::native::vectorized_elementwise_kernel<4, ...>", None),
    ("lcsm::k_fft_spectra<1024>", None),
])
def test_kernel_key(name, key):
    assert bench.kernel_key(name) == key


def _row(i, name, kib):
    return {"Dispatch_Id": str(i), "Kernel_Name": name, "Counter_Value": str(kib)}


def test_tile_bytes_sums_a_column_tile_with_its_red_cell():
    """Dispatch order of two positions: a fused step; then the red cell and
    two column chunks (transpose, transform, transpose each) of the U = 4096
    tile; then a fused step and a wide-panel FFT tile.  The column tile's
    entry is the red cell plus its six dispatches; the other launches stay
    separate; rows arrive out of order and are sorted by dispatch id."""
    order = [
        ("lcsm::k_step_fused<1, true>", 1.0),
        ("lcsm::k_step_fused<0, true>", 0.5),
        ("lcsm::k_rows_to_cols", 20.0),
        ("lcsm::k_fft_coltile<8192>", 100.0),
        ("lcsm::k_cols_to_rows<false>", 30.0),
        ("lcsm::k_rows_to_cols", 21.0),
        ("lcsm::k_fft_coltile<8192>", 101.0),
        ("lcsm::k_cols_to_rows<false>", 31.0),
        ("lcsm::k_step_fused<1, true>", 2.0),
        ("lcsm::k_fft_tile<256, true, true, false, 8>", 7.0),
    ]
    rows = [_row(i, n, v) for i, (n, v) in enumerate(order)]
    per = bench.tile_bytes(rows[::-1])
    assert per[("fft_col", 4096)] == [1024.0 * (0.5 + 20 + 100 + 30 + 21 + 101 + 31)]
    assert per[("fused", 1)] == [1024.0, 2048.0]
    assert per[("fft_lds", 128)] == [7 * 1024.0]
    assert ("red", 0) not in per


def test_tile_bytes_groups_a_mirrored_tile_with_its_copies():
    """A mirrored tile launch: the red cell, the mirror's input copy, the
    transform and the merge are one entry; a following fused step stays apart."""
    order = [("lcsm::k_step_fused<0, true>", 0.5), ("lcsm::k_cm_yin4", 8.0),
             ("lcsm::k_cm_tile<2048>", 40.0), ("lcsm::k_cm_merge4<true>", 9.0),
             ("lcsm::k_step_fused<1, true>", 1.0)]
    per = bench.tile_bytes([_row(i, n, v) for i, (n, v) in enumerate(order)])
    assert per[("fft_cm", 1024)] == [1024.0 * (0.5 + 8 + 40 + 9)]
    assert per[("fused", 1)] == [1024.0]


def test_tile_bytes_three_pass_tile_after_a_mirror_copy():
    """At a multiple of the mirror's T0 whose tile is a three-pass one (2U =
    131072 = 32 x 4096): the red cell, the mirror's input copy and every
    chunk's three passes are one launch of U = 65536."""
    order = [("lcsm::k_step_fused<0, true>", 0.5), ("lcsm::k_cm_yin4", 8.0),
             ("lcsm::k_fft_rows_fwd<4096, true>", 10.0), ("lcsm::k_fft_mid_tile<32>", 11.0),
             ("lcsm::k_fft_rows_inv<4096, false>", 12.0), ("lcsm::k_fft_rows_fwd<4096, true>", 10.0),
             ("lcsm::k_fft_mid_tile<32>", 11.0), ("lcsm::k_fft_rows_inv<4096, false>", 12.0),
             ("lcsm::k_step_fused<1, true>", 1.0)]
    per = bench.tile_bytes([_row(i, n, v) for i, (n, v) in enumerate(order)])
    assert per[("fft_hbm", 65536)] == [1024.0 * (0.5 + 8 + 2 * (10 + 11 + 12))]
    assert per[("fused", 1)] == [1024.0]
    assert not any(k[1] is None for k in per)


def test_tile_bytes_keeps_a_lone_red_cell():
    rows = [_row(1, "lcsm::k_step_fused<0, true>", 0.25),
            _row(2, "lcsm::k_fft_tile<8192, false, true, false>", 50.0)]
    per = bench.tile_bytes(rows)
    assert per[("red", 0)] == [256.0]
    assert per[("fft_lds", 4096)] == [50 * 1024.0]


def test_launch_bytes_hand_counted():
    """One layer, B = 1, D = 2 (2 columns): red cell 16 B per column; a
    fused U = 2 step adds 4 (U - 1) + 8U per column and 4 (2U - 1) lags per
    channel; an FFT tile of U = 4 adds 4 (U - 1) + 8U per column and
    8 (U + 1) spectrum bytes per channel."""
    w = datagen.Workload("hand", 1, 1, 2, 64, decay=1.0, seed=0)
    assert bench.launch_bytes("red", 0, w) == 2 * 16
    assert bench.launch_bytes("fused", 2, w) == 2 * (16 + 4 + 16) + 2 * 4 * 3
    assert bench.launch_bytes("fft_lds", 4, w) == 2 * (16 + 12 + 32) + 2 * 8 * 5


def test_source_digest_files_exist_and_change_with_content(tmp_path, monkeypatch):
    csrc = os.path.join(ROOT, "paper_2410_12982_amd", "csrc")
    for f in bench.COUNTED_SOURCES:
        assert os.path.isfile(os.path.join(csrc, f)), f
    d0 = bench.source_digest()
    assert len(d0) == 16 and d0 == bench.source_digest()
    # the same digest over a copy, then over the copy with one byte changed
    fake = tmp_path / "paper_2410_12982_amd" / "csrc"
    fake.mkdir(parents=True)
    for f in bench.COUNTED_SOURCES:
        with open(os.path.join(csrc, f), "rb") as src:
            (fake / f).write_bytes(src.read())
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.source_digest() == d0
    p = fake / bench.COUNTED_SOURCES[0]
    p.write_bytes(p.read_bytes() + b" ")
    assert bench.source_digest() != d0


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_group_kernels_picks_the_dispatches_of_one_launch():
    """The counter evidence quoted beside the roofline covers exactly the
    dispatches one launch of (kind, U) is made of."""
    g = bench.group_kernels("fft_cm", 1024)
    assert g("k_cm_tile<2048>") and g("k_cm_yin4") and g("k_cm_merge4<true>") and g("k_cm_yin")
    assert not g("k_cm_tile<4096>") and not g("k_fft_tile<2048, true, true, false, 8>")
    assert bench.group_kernels("fft_cm", 16384)("k_cm_tile2<16384, 0>")
    g = bench.group_kernels("fft_lds", 512)
    assert g("k_fft_tile<1024, true, true, false, 8>") and not g("k_fft_tile<128, true, true, false, 8>")
    g = bench.group_kernels("fused", 1)
    assert g("k_step_fused<1, true>") and not g("k_step_fused<16, true>")
    g = bench.group_kernels("fft_hbm", 32768)
    assert g("k_fft_rows_fwd<1024, false>") and g("k_fft_mid_tile<16>") and not g("k_cm_yin4")


def test_trace_summary_names_its_file_and_reports_block_launches(tmp_path, monkeypatch):
    """A closed-loop trace is written under its own name, with the chained-step
    block launches (every instantiation) per launch and per position of the
    one generation."""
    import types
    csrc = os.path.join(ROOT, "paper_2410_12982_amd", "csrc")
    fake = tmp_path / "paper_2410_12982_amd" / "csrc"
    fake.mkdir(parents=True)
    for f in bench.COUNTED_SOURCES:
        with open(os.path.join(csrc, f), "rb") as src:
            (fake / f).write_bytes(src.read())
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    tr = tmp_path / "trace"
    tr.mkdir()
    rows = ["Kernel_Name,Start_Timestamp,End_Timestamp"]
    t = 1000
    for us, tpl in ((10, ""), (12, "<false>"), (14, "<true>")):
        rows.append(f'"void lcsm::(anonymous namespace)::k_chain_block{tpl}(float const*, int)",{t},'
                    f'{t + us * 1000}')
        t += 100000
    rows.append(f'"void lcsm::(anonymous namespace)::k_step_fused<32, false>(float const*)",{t},{t + 5000}')
    (tr / "run_kernel_trace.csv").write_text("\n".join(rows) + "\n")
    args = types.SimpleNamespace(trace_from=str(tr), workload="m1b1d16l1k", command="python3 bench.py",
                                 bracket="", trace_name="closedloop")
    bench.trace_summary(args)
    out = (tmp_path / "profiles" / "closedloop_m1b1d16l1k.txt").read_text()
    assert "3 launches, 12.00 us each" in out
    assert f"{1024 / 3:.2f} positions per launch" in out
    assert f"{36 / 1024:.3f} us of block launch per position" in out
    assert not (tmp_path / "profiles" / "kernels_m1b1d16l1k.txt").exists()


def test_generation_bytes_hand_counted():
    """L = 4, one column: red cells 4 x 16 B; tiles i = 1 (U = 1: 8 B of
    destination, lag 1), i = 2 (U = 2: one more input, 2 destination rows,
    lags 1..3), i = 3 (U = 1).  28 + 48 + 28 + 16 = 120 B."""
    w = datagen.Workload("tiny", 1, 1, 1, 4, decay=1.0, seed=0)
    assert bench.generation_bytes(w) == 120
    # the per-launch figures summed over the positions of a power-of-two run
    w = datagen.Workload("small", 2, 3, 5, 64, decay=1.0, seed=0)
    per = sum(bench.launch_bytes("fused", (t + 1) & -(t + 1), w) for t in range(w.L - 1))
    assert bench.generation_bytes(w) == per + bench.launch_bytes("fused", 0, w)


def test_dd_generation_bytes_hand_counted():
    """L = 4, one column: red cells 4 x 24 B; t = 1 the square of U = 1
    (two inputs, destination row 2: 16 B); t = 2 the tile of U = 1 (four
    inputs, destination row 3: 24 B); t = 3 tiles whose rows lie past L
    (nothing).  96 + 16 + 24 = 136 B."""
    w = datagen.Workload("tiny", 1, 1, 1, 4, decay=1.0, seed=0)
    assert bench.dd_generation_bytes(w) == 136
    w2 = datagen.Workload("tiny2", 2, 3, 5, 4, decay=1.0, seed=0)
    assert bench.dd_generation_bytes(w2) == 136 * 30


def test_generation_roofline_arithmetic():
    r = bench.generation_roofline(8e9, 2.0)     # 8 GB in 2 ms
    assert r == {"algorithmic_GB": 8.0, "GB_s": 4000.0, "frac_of_8TB_s": 0.5}


def test_limiter_of_classifies_by_vector_alu_busy():
    c = {"source": "x", "kernels": {"k_cm_tile<2048>": {"VALUBusy": 87.2}, "k_cm_yin4": {"VALUBusy": 6.9}}}
    got = bench.limiter_of(c)
    assert got["k_cm_tile<2048>"].startswith("vector ALU") and "87.2" in got["k_cm_tile<2048>"]
    assert got["k_cm_yin4"].startswith("memory")
    assert bench.limiter_of(None) is None
