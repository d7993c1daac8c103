"""GPU parity of the prompt prefill (lcsm_prefill; needs an MI355X).

With all P prompt inputs known, the prompt's outputs come from one 2P-point
transform (the filter delayed by P rows), and the context is left exactly as
P online steps would leave it; the generation then continues step by step.
Bars: the whole run (prompt plus generation) against the fp64 static-FFT
oracle on the same teacher-forced inputs, max|z_gpu - z_ref| <= 1e-4 *
max|z_ref|; on small-integer data the rounded outputs equal the exact int64
convolution.
"""
import numpy as np
import pytest
import torch

import datagen
from oracle import conv
from oracle.relaxed import filters_to_columns

from gpu_harness import TOL, dev, lcsm_mod, make_ctx, rel_err, say

pytestmark = pytest.mark.gpu

OPTIONS = {
    "default": None,
    # every tile above U = 1 is an FFT tile, one LDS pass up to 2U = 4096
    "fft_from_2": {"direct_max_u": 1, "lds_fft_max_n": 4096, "col_fft_min_n": 1 << 20},
    # every tile with 2U > 16 (and the prompt's transform) in three passes
    "multipass_from_16": {"direct_max_u": 1, "lds_fft_max_n": 16, "col_fft_min_n": 1 << 20},
    # every FFT tile (and the prompt's transform) on transposed column chunks
    "col_from_4": {"direct_max_u": 1, "col_fft_min_n": 4},
    "colT_from_4": {"direct_max_u": 1, "col_fft_min_n": 4, "col_tile_form": 1},
}


def _prefill_then_run(ctx, y, P):
    z = torch.full_like(y, float("nan"))
    ctx.prefill(y[:P], z[:P])
    assert ctx.position == P
    if y.shape[0] > P:
        ctx.run(y[P:], z[P:])
    torch.cuda.synchronize()
    return z.cpu().numpy()


@pytest.mark.parametrize("opt", ["default", "fft_from_2", "multipass_from_16", "col_from_4",
                                 "colT_from_4"])
@pytest.mark.parametrize("case", [(2, 3, 40, 1024, 256), (3, 2, 33, 2048, 64), (1, 1, 5, 300, 128),
                                  (2, 2, 24, 4096, 2048), (1, 2, 8, 32768, 16384)])
def test_prefill_then_generate_matches_oracle(opt, case):
    """The last case's prompt tile is 2U = 32768: with column tiles it runs as
    the two 16384-point halves, with the filter spectrum delayed by P."""
    M, B, D, L, P = case
    w = datagen.Workload("prefill", M, B, D, L, decay=L / 4, seed=31 + P)
    say(f"[prefill] M={M} B={B} D={D} L={L} P={P} options={opt}")
    ctx, _ = make_ctx(w, options=OPTIONS[opt])
    y = datagen.y_torch(w, dev())
    z = _prefill_then_run(ctx, y, P)
    h = filters_to_columns(datagen.filters_np(w), w.B)
    zr = conv.causal_conv_fft(y.cpu().numpy().reshape(L, -1).astype(np.float64), h.reshape(h.shape[0], -1))
    err_prompt = rel_err(z[:P].reshape(P, -1), zr[:P])
    err = rel_err(z.reshape(L, -1), zr)
    say(f"  rel err prompt {err_prompt:.3e}, whole run {err:.3e}")
    assert err <= TOL


def test_prefill_bench_workload_half_prompt():
    """m1b8d768l8k with a 4096-position prompt (the 2U = 8192 transform for
    the prompt's outputs), then 4096 online steps."""
    w = datagen.WORKLOADS["m1b8d768l8k"]
    P = w.L // 2
    say(f"[prefill] {w.name} P={P}")
    ctx, _ = make_ctx(w)
    y = datagen.y_torch(w, dev())
    z = _prefill_then_run(ctx, y, P)
    h = filters_to_columns(datagen.filters_np(w), w.B)
    zr = conv.causal_conv_fft(y.cpu().numpy().reshape(w.L, -1).astype(np.float64), h.reshape(h.shape[0], -1))
    err = rel_err(z.reshape(w.L, -1), zr)
    say(f"  rel err {err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("opt", ["default", "multipass_from_16", "col_from_4"])
def test_prefill_integer_data_rounds_to_exact(opt):
    M, B, D, L, P = 2, 2, 16, 2048, 512
    w = datagen.Workload("int", M, B, D, L, decay=1.0, seed=7)
    h = datagen.int_filters_np(w, 3)
    y = datagen.int_y_np(w, 3)
    say(f"[prefill int] M={M} B={B} D={D} L={L} P={P} options={opt}")
    ctx, _ = make_ctx(w, torch.from_numpy(h).to(dev()), OPTIONS[opt])
    z = _prefill_then_run(ctx, torch.from_numpy(y).to(dev()), P)
    ex = np.zeros((L, M, B, D), dtype=np.int64)
    hi, yi = h.astype(np.int64), y.astype(np.int64)
    for k in range(L):
        ex[k:] += yi[: L - k] * hi[None, :, None, :, k]
    assert np.abs(z.astype(np.float64) - ex).max() < 0.25
    assert np.array_equal(np.rint(z).astype(np.int64), ex)


def test_prefill_continues_like_stepwise_run_and_reset_repeats():
    """Prefill + steps against all steps on the same inputs (the two orders of
    summation agree to fp32 rounding), and a reset context prefills again to
    the same bits."""
    w = datagen.Workload("prefill2", 2, 2, 48, 2048, decay=512.0, seed=5)
    P = 512
    ctx, _ = make_ctx(w)
    y = datagen.y_torch(w, dev())
    za = _prefill_then_run(ctx, y, P)
    ctx.reset()
    zb = torch.empty_like(y)
    ctx.run(y, zb)
    torch.cuda.synchronize()
    zb = zb.cpu().numpy()
    assert rel_err(za, zb.astype(np.float64)) <= 1e-5
    ctx.reset()
    zc = _prefill_then_run(ctx, y, P)
    assert np.array_equal(za, zc)


def test_prefill_errors():
    lcsm = lcsm_mod()
    w = datagen.Workload("prefill3", 1, 1, 8, 256, decay=64.0, seed=3)
    ctx, _ = make_ctx(w)
    y = datagen.y_torch(w, dev())
    z = torch.empty_like(y)
    for P in (0, 3, 96, 256):  # not a power of two, or 2P > L
        with pytest.raises(lcsm.LcsmError) as ex:
            ctx.prefill(y[:max(P, 1)] if P else y[:1], z, P=P)
        assert ex.value.code == lcsm.LCSM_EINVAL
    ctx.step(y[0], z[0])
    with pytest.raises(lcsm.LcsmError) as ex:
        ctx.prefill(y[:64], z[:64])
    assert ex.value.code == lcsm.LCSM_ESTATE
    ctx.reset()
    ctx.prefill(y[:128], z[:128])
    assert ctx.position == 128
