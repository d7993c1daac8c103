"""GPU parity of the FFT gray tiles (needs an MI355X).

The tiles with U above the crossover run as 2U-point cyclic FFT
convolutions with precomputed filter spectra (Lemma 1, App. B): in one LDS
pass when 2U fits, else in three passes through a chunked scratch buffer.
The option sets below force each form onto every tile size a short run has,
including ragged column counts (odd B*D, D not a multiple of the panel
width) and a scratch cap small enough to need many chunks.

Bars: on small-integer data the exact result is an integer and the fp32
FFT error stays far below 1/2, so the rounded GPU output must equal the
exact int64 convolution; on random data max|z_gpu - z_ref| <= 1e-4 *
max|z_ref| against the fp64 oracle.
"""
import numpy as np
import pytest
import torch

import datagen
from oracle import conv, feedback
from oracle.relaxed import filters_to_columns, relaxed_online

from gpu_harness import TOL, dev, lcsm_mod, make_ctx, rel_err, say, say_maxima

pytestmark = pytest.mark.gpu

FFT_OPTIONS = {
    # every tile with U >= 2 is an FFT tile, in one LDS pass up to 2U = 4096
    "lds_from_2": {"direct_max_u": 1, "lds_fft_max_n": 4096, "col_fft_min_n": 1 << 20},
    # every tile with 2U > 16 goes through the three-pass form
    "multipass_from_16": {"direct_max_u": 1, "lds_fft_max_n": 16, "col_fft_min_n": 1 << 20},
    # multi-pass with a 1 MiB scratch: many chunks per tile
    "tiny_scratch": {"direct_max_u": 4, "lds_fft_max_n": 32, "scratch_mib": 1, "col_fft_min_n": 1 << 20},
    # every FFT tile on the column-major mirror (the column path is off above):
    # T0 = 2, a merge after every other position
    "col_from_4": {"direct_max_u": 1, "col_fft_min_n": 4},
    # the same tiles on transposed column chunks
    "colT_from_4": {"direct_max_u": 1, "col_fft_min_n": 4, "col_tile_form": 1},
    # column tiles with a 1 MiB scratch: many column chunks per tile (transposed),
    # many pair chunks of the split 2U = 32768 tile (mirror)
    "col_tiny_scratch": {"direct_max_u": 4, "col_fft_min_n": 16, "scratch_mib": 1},
    "colT_tiny_scratch": {"direct_max_u": 4, "col_fft_min_n": 16, "scratch_mib": 1,
                          "col_tile_form": 1},
    "default": None,
}


def _int_case(M, B, D, L, r, seed):
    w = datagen.Workload("int", M, B, D, L, decay=1.0, seed=seed)
    return w, datagen.int_filters_np(w, r), datagen.int_y_np(w, r)


def _exact(h, y):
    L, M, B, D = y.shape
    z = np.zeros((L, M, B, D), dtype=np.int64)
    for m in range(M):
        for b in range(B):
            for d in range(D):
                z[:, m, b, d] = np.convolve(y[:, m, b, d].astype(np.int64),
                                            h[m, d].astype(np.int64))[:L]
    return z


def _run_full(ctx, y):
    z = torch.empty_like(y)
    ctx.run(y, z)
    torch.cuda.synchronize()
    return z.cpu().numpy()


@pytest.mark.parametrize("opt", ["lds_from_2", "multipass_from_16", "tiny_scratch", "col_from_4",
                                 "col_tiny_scratch", "colT_from_4", "colT_tiny_scratch"])
@pytest.mark.parametrize("shape", [(2, 3, 40, 300), (1, 1, 5, 257), (3, 2, 33, 1000),
                                   (1, 4, 64, 2048)])
def test_integer_data_rounds_to_exact(opt, shape):
    M, B, D, L = shape
    say(f"[int fft] M={M} B={B} D={D} L={L} options={opt}")
    w, h, y = _int_case(M, B, D, L, 3, seed=3 * sum(shape))
    ctx, _ = make_ctx(w, torch.from_numpy(h).to(dev()), FFT_OPTIONS[opt])
    z = _run_full(ctx, torch.from_numpy(y).to(dev()))
    ex = _exact(h, y)
    err = np.abs(z.astype(np.float64) - ex).max()
    say(f"  max abs err {err:.3e}")
    assert err < 0.25
    assert np.array_equal(np.rint(z).astype(np.int64), ex)


@pytest.mark.parametrize("opt", ["default", "lds_from_2", "col_from_4", "colT_from_4"])
@pytest.mark.parametrize("shape", [(1, 2, 48, 4500), (1, 3, 24, 4200), (2, 1, 10, 6000)])
def test_integer_data_panel_orders_and_clipped_large_tiles(opt, shape):
    """Shapes whose channel count is not a whole number of 128-byte line
    groups of panels (48 and 24 channels: the batch-row panel order), or not
    a whole number of panels (10 channels), and lengths that clip the 2U =
    8192 tile's destination window (the general, bounds-checked kernel)."""
    M, B, D, L = shape
    say(f"[int fft panels/clipped] M={M} B={B} D={D} L={L} options={opt}")
    w, h, y = _int_case(M, B, D, L, 3, seed=5 * sum(shape))
    ctx, _ = make_ctx(w, torch.from_numpy(h).to(dev()), FFT_OPTIONS[opt])
    z = _run_full(ctx, torch.from_numpy(y).to(dev()))
    ex = _exact(h, y)
    err = np.abs(z.astype(np.float64) - ex).max()
    say(f"  max abs err {err:.3e}")
    assert err < 0.25
    assert np.array_equal(np.rint(z).astype(np.int64), ex)


@pytest.mark.parametrize("half", [False, True])
@pytest.mark.parametrize("opt", ["default", "lds_from_2"])
@pytest.mark.parametrize("shape", [(1, 2, 8192, 260), (2, 3, 2731, 200), (1, 5, 3300, 140)])
def test_integer_data_wide_panels(opt, shape, half):
    """From 2^14 columns the single-pass tiles of 2U = 128 and 256 use panels
    of 8 complex columns: whole panels inside a batch row (8192 channels),
    an odd column count per layer (2731 channels, 3 batch rows), channels
    not a whole number of panels (3300), a clipped destination (L = 260 cuts
    the U = 128 tile of i = 256), and, with half-state storage, the in-place
    tile of i = T = 128 at 2U = 256."""
    M, B, D, L = shape
    say(f"[int fft wide panels] M={M} B={B} D={D} L={L} options={opt} half_state={half}")
    w, h, y = _int_case(M, B, D, L, 3, seed=7 * sum(shape))
    opts = dict(FFT_OPTIONS[opt] or {})
    if half:
        opts["half_state"] = 1
    ctx, _ = make_ctx(w, torch.from_numpy(h).to(dev()), opts or None)
    z = _run_full(ctx, torch.from_numpy(y).to(dev()))
    ex = _exact(h, y)
    err = np.abs(z.astype(np.float64) - ex).max()
    say(f"  max abs err {err:.3e}")
    assert err < 0.25
    assert np.array_equal(np.rint(z).astype(np.int64), ex)


@pytest.mark.parametrize("half", [False, True])
@pytest.mark.parametrize("opt", ["col_from_4", "col_tiny_scratch", "colT_from_4", "colT_tiny_scratch"])
@pytest.mark.parametrize("shape", [(2, 3, 40, 301), (1, 2, 64, 1027), (1, 1, 12, 1028)])
def test_integer_data_column_transposes(opt, shape, half):
    """Column tiles whose transposes move 16-byte vectors (B*D a multiple of
    4) next to clipped destinations of a length that is not (L = 301 and
    1027: the outputs go back element by element), and, with half-state
    storage, the in-place tile of i = T with both kinds of destination
    (45 rows at L = 301, 4 rows at L = 1028)."""
    M, B, D, L = shape
    say(f"[int fft column transposes] M={M} B={B} D={D} L={L} options={opt} half_state={half}")
    w, h, y = _int_case(M, B, D, L, 3, seed=11 * sum(shape))
    opts = dict(FFT_OPTIONS[opt], half_state=int(half))
    ctx, _ = make_ctx(w, torch.from_numpy(h).to(dev()), opts)
    z = _run_full(ctx, torch.from_numpy(y).to(dev()))
    ex = _exact(h, y)
    err = np.abs(z.astype(np.float64) - ex).max()
    say(f"  max abs err {err:.3e}")
    assert err < 0.25
    assert np.array_equal(np.rint(z).astype(np.int64), ex)


@pytest.mark.parametrize("half", [False, True])
@pytest.mark.parametrize("opt", ["col_from_4", "col_top", "colT_top"])
@pytest.mark.parametrize("shape", [(1, 4, 16, 16500), (1, 1, 64, 17000), (1, 1, 5, 16390)])
def test_integer_data_split_column_tile(opt, shape, half):
    """The column tile of 2U = 32768 (i = 16384, clipped at L), transformed as
    its even and odd bins in two 16384-point halves: batch-row pairs of one
    channel (B*D = 64, B even), channel pairs (B = 1), neighbouring columns
    with an odd count; every FFT tile on column chunks or only this one; with
    half-state storage it is the in-place tile of i = T = 16384."""
    M, B, D, L = shape
    say(f"[int split column tile] M={M} B={B} D={D} L={L} options={opt} half_state={half}")
    w, h, y = _int_case(M, B, D, L, 2, seed=13 * sum(shape))
    top = {"col_top": {"col_fft_min_n": 32768},
           "colT_top": {"col_fft_min_n": 32768, "col_tile_form": 1}}
    opts = dict(FFT_OPTIONS[opt] if opt in FFT_OPTIONS else top[opt], half_state=int(half))
    ctx, _ = make_ctx(w, torch.from_numpy(h).to(dev()), opts)
    lcsm = lcsm_mod()
    form = lcsm.TILE_FFT_COL if (half or opts.get("col_tile_form")) else lcsm.TILE_FFT_CM
    assert ctx.tile(16383)[1:] == (16384, L - 16384, form)
    z = _run_full(ctx, torch.from_numpy(y).to(dev()))
    # the exact integers: the oracle's fp64 FFT convolution, rounded (|z| stays
    # near 10^3, where fp64 rounding is far below 1/2)
    hc = filters_to_columns(h.astype(np.float64), B).reshape(L, -1)
    zf = conv.causal_conv_fft(y.reshape(L, -1).astype(np.float64), hc)
    ex = np.rint(zf).astype(np.int64)
    assert np.abs(zf - ex).max() < 1e-3
    ex = ex.reshape(L, M, B, D)
    err = np.abs(z.astype(np.float64) - ex).max()
    say(f"  max abs err {err:.3e}")
    assert err < 0.25
    assert np.array_equal(np.rint(z).astype(np.int64), ex)


@pytest.mark.parametrize("opt", ["lds_from_2", "multipass_from_16", "tiny_scratch", "default",
                                 "col_from_4"])
def test_m1b8d768l8k_teacher_forced_all_columns(opt):
    w = datagen.WORKLOADS["m1b8d768l8k"]
    say(f"[fft teacher-forced all columns] {w.name} options={opt}")
    ctx, _ = make_ctx(w, options=FFT_OPTIONS[opt])
    y = datagen.y_torch(w, dev())
    z = _run_full(ctx, y)
    h = filters_to_columns(datagen.filters_np(w), w.B)
    zr = conv.causal_conv_fft(y.cpu().numpy().reshape(w.L, -1).astype(np.float64), h[:, 0])
    err = rel_err(z.reshape(w.L, -1), zr)
    say(f"  rel err {err:.3e}")
    cols = np.array([(m, b, d) for m in range(w.M) for b in range(w.B) for d in range(w.D)])
    say_maxima(z.reshape(w.L, -1), zr, cols)
    assert err <= TOL


@pytest.mark.parametrize("opt", ["lds_from_2", "multipass_from_16"])
def test_small_workload_closed_loop(opt):
    w = datagen.WORKLOADS["m1b1d16l1k"]
    say(f"[fft closed loop] {w.name} options={opt}")
    ctx, _ = make_ctx(w, options=FFT_OPTIONS[opt])
    x = datagen.x_torch(w, dev())
    z = torch.empty_like(x)
    for t in range(w.L):
        ctx.step_chain(x[t], z[t])
    torch.cuda.synchronize()
    h = filters_to_columns(datagen.filters_np(w), w.B)
    zr, _ = relaxed_online(h, feedback.tanh_chain(datagen.x_np(w).reshape(w.L, w.M, -1), w.M))
    err = rel_err(z.cpu().numpy().reshape(w.L, w.M, -1), zr)
    say(f"  closed-loop rel err {err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("opt", ["default", "multipass_from_16", "col_tiny_scratch"])
def test_fft_rerun_bitwise_and_step_layer_path(opt):
    w = datagen.Workload("fftdet", 3, 2, 70, 1500, decay=400.0, seed=12)
    say(f"[fft determinism / step_layer] M=3 B=2 D=70 L=1500 options={opt}")
    ctx, filt = make_ctx(w, options=FFT_OPTIONS[opt])
    y = datagen.y_torch(w, dev())
    z1 = _run_full(ctx, y)
    ctx.reset()
    z2 = _run_full(ctx, y)
    assert np.array_equal(z1, z2)
    ctx.reset()
    z3 = torch.empty_like(y)
    for t in range(w.L):
        for m in range(w.M):
            ctx.step_layer(m, y[t, m], z3[t, m])
        ctx.advance()
    torch.cuda.synchronize()
    assert np.array_equal(z1, z3.cpu().numpy())
    h = filters_to_columns(datagen.filters_np(w), w.B)
    yn = y.cpu().numpy().reshape(w.L, w.M, -1).astype(np.float64)
    zr = conv.causal_conv_fft(yn, h)
    assert rel_err(z1.reshape(w.L, w.M, -1), zr) <= TOL


@pytest.mark.parametrize("opt", ["default", "multipass_from_16"])
def test_fft_causality_past_outputs_bit_identical(opt):
    w = datagen.Workload("causal", 2, 2, 96, 1000, decay=300.0, seed=8)
    say(f"[fft causality] M=2 B=2 D=96 L=1000 options={opt}")
    ctx, _ = make_ctx(w, options=FFT_OPTIONS[opt])
    y1 = datagen.y_torch(w, dev())
    y2 = y1.clone()
    t0 = 511
    y2[t0 + 1:] = -y2[t0 + 1:] * 0.5
    z1 = _run_full(ctx, y1)
    ctx.reset()
    z2 = _run_full(ctx, y2)
    assert np.array_equal(z1[: t0 + 1], z2[: t0 + 1])
    assert not np.array_equal(z1[t0 + 1:], z2[t0 + 1:])


def test_geometric_filter_multipass():
    """h = r^k (one-state LTI system): z_t = r z_{t-1} + y_t, through the
    three-pass tiles at every U >= 16."""
    M, B, D, L = 1, 1, 32, 8192
    say(f"[geometric multipass] M={M} B={B} D={D} L={L}")
    w = datagen.Workload("geo", M, B, D, L, decay=1.0, seed=10)
    r = (0.9 + 0.0995 * np.linspace(0, 1, M * D).reshape(M, D)).astype(np.float32).astype(np.float64)
    h = (r[:, :, None] ** np.arange(L)[None, None, :]).astype(np.float32)
    ctx, _ = make_ctx(w, torch.from_numpy(h).to(dev()), FFT_OPTIONS["multipass_from_16"])
    y = datagen.y_torch(w, dev())
    z = _run_full(ctx, y)
    yn = y.cpu().numpy().astype(np.float64)
    zr = conv.geometric_recurrence(yn[:, 0], r[0][None, :])
    assert rel_err(z[:, 0], zr) <= TOL
