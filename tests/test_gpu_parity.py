"""GPU parity of the HIP library against the CPU oracle (needs an MI355X).

Every case drives the library through its C ABI (ctypes binding) and compares
element by element with the fp64 oracle on the same seeded inputs.  Bars:
bit-exact on small-integer data (all partial sums are exact in fp32), else
max|z_gpu - z_ref| <= 1e-4 * max|z_ref|.
"""
import numpy as np
import pytest
import torch

import datagen
from oracle import conv, feedback
from oracle.relaxed import filters_to_columns, relaxed_online

from gpu_harness import TOL, dev, lcsm_mod, make_ctx, oracle_sampled, rel_err, run_sampled, say

pytestmark = pytest.mark.gpu

# direct kernels only / crossover into FFT tiles (single LDS pass and multi-pass)
OPTION_SETS = {
    "all_direct": {"direct_max_u": 1 << 20},
    "default": None,
    "fft_from_2": {"direct_max_u": 1, "lds_fft_max_n": 64, "col_fft_min_n": 1 << 20},
    "fft_from_64": {"direct_max_u": 32},
}


def _int_case(M, B, D, L, r, seed):
    w = datagen.Workload("int", M, B, D, L, decay=1.0, seed=seed)
    h = datagen.int_filters_np(w, r)
    y = datagen.int_y_np(w, r)
    return w, h, y


def _exact(h, y):
    """Exact integer reference z[t, m, b, d] via np.convolve in int64."""
    L, M, B, D = y.shape
    z = np.zeros((L, M, B, D), dtype=np.int64)
    hi = h.astype(np.int64)
    yi = y.astype(np.int64)
    for m in range(M):
        for b in range(B):
            for d in range(D):
                z[:, m, b, d] = np.convolve(yi[:, m, b, d], hi[m, d])[:L]
    return z


def _run_full(ctx, y):
    z = torch.empty_like(y)
    ctx.run(y, z)
    torch.cuda.synchronize()
    return z.cpu().numpy()


@pytest.mark.parametrize("shape", [(2, 3, 40, 300), (1, 2, 64, 256), (3, 1, 5, 1), (1, 1, 1, 77),
                                   (2, 2, 300, 129), (1, 4, 8200, 100), (2, 3, 5462, 70)])
def test_integer_data_bit_exact_direct(shape):
    """The last two shapes have more than 2^15 columns, channel counts that
    leave a partial block of 256, and clipped direct tiles (i = 96 at L = 100:
    4 rows; i = 64 at L = 70: 6 rows)."""
    M, B, D, L = shape
    say(f"[int-exact direct] M={M} B={B} D={D} L={L}")
    w, h, y = _int_case(M, B, D, L, 3, seed=sum(shape))
    ctx, _ = make_ctx(w, torch.from_numpy(h).to(dev()), OPTION_SETS["all_direct"])
    z = _run_full(ctx, torch.from_numpy(y).to(dev()))
    assert np.array_equal(z.astype(np.int64), _exact(h, y))


def test_step_layer_path_equals_step_path():
    M, B, D, L = 3, 2, 70, 200
    say(f"[step_layer vs step] M={M} B={B} D={D} L={L}")
    w, h, y = _int_case(M, B, D, L, 3, seed=5)
    hf = torch.from_numpy(h).to(dev())
    yd = torch.from_numpy(y).to(dev())
    ctx, _ = make_ctx(w, hf, OPTION_SETS["all_direct"])
    z1 = _run_full(ctx, yd)
    ctx2, _ = make_ctx(w, hf, OPTION_SETS["all_direct"])
    z2 = torch.empty_like(yd)
    for t in range(L):
        for m in range(M):
            ctx2.step_layer(m, yd[t, m], z2[t, m])
        ctx2.advance()
    torch.cuda.synchronize()
    assert np.array_equal(z1, z2.cpu().numpy())


def test_small_workload_teacher_forced():
    w = datagen.WORKLOADS["m1b1d16l1k"]
    say(f"[teacher-forced] {w.name}")
    ctx, _ = make_ctx(w)
    y = datagen.y_torch(w, dev())
    z = _run_full(ctx, y)
    h = filters_to_columns(datagen.filters_np(w), w.B)         # [L, M, B*D]
    zr = conv.causal_conv_naive(y.cpu().numpy().reshape(w.L, w.M, -1), h)
    assert rel_err(z.reshape(w.L, w.M, -1), zr) <= TOL


def test_small_workload_closed_loop():
    """The full online problem: the tanh chain feeds z_t back into y_{t+1}."""
    w = datagen.WORKLOADS["m1b1d16l1k"]
    say(f"[closed loop] {w.name}")
    ctx, _ = make_ctx(w)
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


@pytest.mark.parametrize("opt", ["default", "fft_from_2", "all_direct"])
@pytest.mark.parametrize("shape", [(4, 2, 24, 300), (11, 1, 8, 130), (18, 1, 8, 100), (33, 1, 4, 70)])
def test_multilayer_closed_loop(opt, shape):
    """The chain across layers (y^m_t from z^{m-1}_t, layer 0 from the last
    layer's z_{t-1}): with several layers the red cells walk the layers in
    chunks of loads (8, 16 or 32 layers: 11 and 18 layers in one chunk, 33 in
    two) and the tiles run in the separate all-layer launch.
    Filters decay fast (as in the 1024-position workload), so the fp32 closed
    loop stays close to the fp64 one over these lengths."""
    M, B, D, L = shape
    w = datagen.Workload("chain", M, B, D, L, decay=200.0, seed=21 + M)
    say(f"[multi-layer closed loop] M={M} B={B} D={D} L={L} options={opt}")
    ctx, _ = make_ctx(w, options=OPTION_SETS[opt])
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


@pytest.mark.parametrize("opt", ["all_direct"])
def test_m1b8d768l8k_teacher_forced_all_columns(opt):
    w = datagen.WORKLOADS["m1b8d768l8k"]
    say(f"[teacher-forced all columns] {w.name} options={opt}")
    ctx, _ = make_ctx(w, options=OPTION_SETS[opt])
    y = datagen.y_torch(w, dev())
    z = _run_full(ctx, y)
    h = filters_to_columns(datagen.filters_np(w), w.B)
    zr = conv.causal_conv_fft(y.cpu().numpy().reshape(w.L, -1).astype(np.float64), h[:, 0])
    err = rel_err(z.reshape(w.L, -1), zr)
    say(f"  rel err {err:.3e}")
    assert err <= TOL


def test_rerun_is_bitwise_deterministic_and_reset_restarts():
    w = datagen.WORKLOADS["m1b8d768l8k"]
    say(f"[determinism/reset] {w.name}")
    ctx, _ = make_ctx(w)
    y = datagen.y_torch(w, dev())
    z1 = _run_full(ctx, y)
    lcsm = lcsm_mod()
    with pytest.raises(lcsm.LcsmError) as e:
        ctx.step(y[0])
    assert e.value.code == lcsm.LCSM_EDONE
    ctx.reset()
    assert ctx.position == 0
    z2 = _run_full(ctx, y)
    assert np.array_equal(z1, z2)


def test_causality_future_inputs_leave_past_outputs_bit_identical():
    w = datagen.Workload("causal", 2, 2, 96, 1000, decay=300.0, seed=8)
    say("[causality] M=2 B=2 D=96 L=1000")
    ctx, _ = make_ctx(w)
    y1 = datagen.y_torch(w, dev())
    y2 = y1.clone()
    t0 = 613
    y2[t0 + 1:] = -y2[t0 + 1:] * 0.5
    z1 = _run_full(ctx, y1)
    ctx.reset()
    z2 = _run_full(ctx, y2)
    assert np.array_equal(z1[: t0 + 1], z2[: t0 + 1])
    assert not np.array_equal(z1[t0 + 1:], z2[t0 + 1:])


@pytest.mark.parametrize("opt", ["all_direct", "default"])
def test_nan_poison_stays_in_its_column_and_reaches_all_later_outputs(opt):
    """A NaN input reaches every later output of its column (coverage >= 1,
    causality).  Direct tiles keep it in that column; FFT tiles carry the
    real columns c and c^1 of a layer together in one complex transform, so
    there it may also reach the partner column, and nothing else."""
    w = datagen.Workload("nan", 2, 3, 50, 512, decay=100.0, seed=9)
    say(f"[nan poison] M=2 B=3 D=50 L=512 options={opt}")
    ctx, _ = make_ctx(w, options=OPTION_SETS[opt])
    y = datagen.y_torch(w, dev())
    t0, col = 123, (1, 2, 17)
    y[t0, col[0], col[1], col[2]] = float("nan")
    z = _run_full(ctx, y)
    zc = z.reshape(w.L, w.M, w.B * w.D)
    c = col[1] * w.D + col[2]
    assert np.all(np.isnan(zc[t0:, col[0], c]))
    mask = np.ones(zc.shape, dtype=bool)
    mask[t0:, col[0], c] = False
    if opt != "all_direct":
        mask[t0:, col[0], c ^ 1] = False
    assert np.all(np.isfinite(zc[mask]))
    assert np.all(np.isfinite(zc[:t0]))


def test_geometric_filter_matches_recurrence():
    """h[m, d, k] = r^k (a one-state LTI system): z_t = r z_{t-1} + y_t."""
    M, B, D, L = 2, 2, 64, 4096
    say(f"[geometric filter] M={M} B={B} D={D} L={L}")
    w = datagen.Workload("geo", M, B, D, L, decay=1.0, seed=10)
    # r is rounded to fp32 first, so the recurrence and the taps use one r
    r = (0.9 + 0.0995 * np.linspace(0, 1, M * D).reshape(M, D)).astype(np.float32).astype(np.float64)
    h = (r[:, :, None] ** np.arange(L)[None, None, :]).astype(np.float32)
    ctx, _ = make_ctx(w, torch.from_numpy(h).to(dev()))
    y = datagen.y_torch(w, dev())
    z = _run_full(ctx, y)
    yn = y.cpu().numpy().astype(np.float64)
    zr = np.empty_like(yn)
    for m in range(M):
        zr[:, m] = conv.geometric_recurrence(yn[:, m], r[m][None, :])
    # the taps are r^k rounded to fp32 one by one (relative 6e-8 each)
    assert rel_err(z, zr) <= TOL


def test_sequencing_errors():
    w = datagen.Workload("seq", 3, 1, 8, 16, decay=4.0, seed=11)
    say("[sequencing] M=3 B=1 D=8 L=16")
    lcsm = lcsm_mod()
    ctx, _ = make_ctx(w)
    y = torch.zeros((w.B, w.D), device=dev())
    with pytest.raises(lcsm.LcsmError) as e:
        ctx.step_layer(1, y)
    assert e.value.code == lcsm.LCSM_ESTATE
    ctx.step_layer(0, y)
    with pytest.raises(lcsm.LcsmError) as e:
        ctx.advance()
    assert e.value.code == lcsm.LCSM_ESTATE
    with pytest.raises(lcsm.LcsmError) as e:
        ctx.step(torch.zeros((w.M, w.B, w.D), device=dev()))
    assert e.value.code == lcsm.LCSM_ESTATE
    ctx.step_layer(1, y)
    ctx.step_layer(2, y)
    ctx.advance()
    assert ctx.position == 1
    with pytest.raises(ValueError):
        ctx.step(torch.zeros((w.M, w.B, w.D + 1), device=dev()))


def _exact_by_lag(h, y):
    """Exact integer reference like _exact, vectorised over columns: one
    shifted multiply-add per lag (z[t] += y[t-k] h[k])."""
    L, M, B, D = y.shape
    hi = h.astype(np.int64)            # [M, D, L]
    yi = y.astype(np.int64)            # [L, M, B, D]
    z = np.zeros_like(yi)
    for k in range(L):
        z[k:] += yi[: L - k] * hi[None, :, None, :, k]
    return z


@pytest.mark.parametrize("opt", ["default", "fft_from_2"])
@pytest.mark.parametrize("shape", [(16384, 1, 1, 64), (1, 65535, 1, 64)])
def test_integer_data_at_the_layer_and_batch_limits(opt, shape):
    """The largest layer count (16384: the step launches are split over layers
    to keep grid z within 65536 blocks) and batch-row count (65535: grid y)
    the library accepts, on small-integer data: bit-exact with direct tiles,
    rounding to the exact integers with FFT tiles (error far below 1/2)."""
    M, B, D, L = shape
    say(f"[limits] M={M} B={B} D={D} L={L} options={opt}")
    w, h, y = _int_case(M, B, D, L, 3, seed=sum(shape))
    ctx, _ = make_ctx(w, torch.from_numpy(h).to(dev()), OPTION_SETS[opt])
    z = _run_full(ctx, torch.from_numpy(y).to(dev()))
    ctx.close()
    ex = _exact_by_lag(h, y)
    if opt == "default":  # every tile of a 64-long run is direct
        assert np.array_equal(z, ex.astype(np.float32))
    else:
        assert np.abs(z.astype(np.float64) - ex).max() < 0.25
        assert np.array_equal(np.rint(z).astype(np.int64), ex)
