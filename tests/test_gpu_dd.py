"""GPU parity of the data-dependent-filter path (include/lcsm_dd.h; needs an
MI355X).

At step t the library receives y_t and rho_t and returns z_t =
sum_{j+k=t} y_j rho_k; the tiles are the parallelogram tiles of Alg. 5 (every
power of two U dividing t+1), direct or as 2U-point FFTs.  Bars: on random
data max|z_gpu - z_ref| <= 1e-4 * max|z_ref| against the fp64 oracle
(oracle/dd.py, itself pinned to the definition); on small-integer data the
rounded outputs equal the exact int64 products; a fixed rho gives the
ordinary convolution.  The option sets put every tile on the direct kernel,
every tile above U = 1 on the FFT kernel, and the default crossover; two
more cap the FFT transform at 16 and 64 points, so that tiles of U = 16 ..
512 run as pairs of 8- or 32-row blocks (up to 64 x 64 pairs, both output
parities, clipped last blocks) -- the form the tiles wider than one LDS
pass take on the 32768- and 131072-position workloads, which are checked
at full size on sampled columns.
"""
import numpy as np
import pytest
import torch

import datagen
from oracle.dd import relaxed_dd

from gpu_harness import TOL, dev, lcsm_mod, rel_err, say

pytestmark = pytest.mark.gpu

OPTIONS = {
    "direct_all": {"direct_max_u": 1 << 20},
    "fft_from_2": {"direct_max_u": 1},
    "default": None,
    "blocks_of_8": {"direct_max_u": 1, "lds_fft_max_n": 16},
    "blocks_of_32": {"direct_max_u": 4, "lds_fft_max_n": 64},
}


def _run(ctx, y, rho):
    z = torch.full_like(y, float("nan"))
    for t in range(y.shape[0]):
        ctx.step(y[t], rho[t], z[t])
    torch.cuda.synchronize()
    return z.cpu().numpy()


def _ctx(w, opt):
    return lcsm_mod().Dd(w.M, w.B, w.D, w.L, options=OPTIONS[opt])


@pytest.mark.parametrize("opt", ["direct_all", "fft_from_2", "default", "blocks_of_8", "blocks_of_32"])
@pytest.mark.parametrize("shape", [(1, 1, 16, 300), (2, 3, 20, 1000), (3, 2, 33, 513),
                                   (1, 4, 64, 2048), (2, 1, 15, 400)])
def test_dd_matches_oracle(opt, shape):
    """Includes an odd column count per layer (15: the FFT tile's last real
    column has no partner in its pair)."""
    M, B, D, L = shape
    say(f"[dd] M={M} B={B} D={D} L={L} options={opt}")
    w = datagen.Workload("dd", M, B, D, L, decay=L / 4, seed=60 + L % 89)
    ctx = _ctx(w, opt)
    y, rho = datagen.y_torch(w, dev()), datagen.rho_torch(w, dev())
    z = _run(ctx, y, rho)
    assert ctx.position == L
    zr = relaxed_dd(y.cpu().numpy().reshape(L, -1), rho.cpu().numpy().reshape(L, -1))
    err = rel_err(z.reshape(L, -1), zr)
    say(f"  rel err {err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("opt", ["direct_all", "fft_from_2", "blocks_of_8"])
def test_dd_integer_data_rounds_to_exact(opt):
    M, B, D, L = 2, 2, 12, 700
    w = datagen.Workload("ddint", M, B, D, L, decay=1.0, seed=3)
    say(f"[dd int] M={M} B={B} D={D} L={L} options={opt}")
    y, rho = datagen.int_y_np(w, 3), datagen.int_rho_np(w, 3)
    ctx = _ctx(w, opt)
    z = _run(ctx, torch.from_numpy(y).to(dev()), torch.from_numpy(rho).to(dev()))
    yi, ri = y.astype(np.int64).reshape(L, -1), rho.astype(np.int64).reshape(L, -1)
    ex = np.zeros((L, yi.shape[1]), dtype=np.int64)
    for k in range(L):
        ex[k:] += yi[: L - k] * ri[k][None, :]
    err = np.abs(z.reshape(L, -1).astype(np.float64) - ex).max()
    say(f"  max abs err {err:.3e}")
    assert err < 0.25
    assert np.array_equal(np.rint(z.reshape(L, -1)).astype(np.int64), ex)


def test_dd_fixed_filter_is_the_convolution_and_reset_repeats():
    """rho_t = h_t, the same for every batch row: the data-independent case,
    against the static FFT convolution of the oracle; a reset context gives
    the same bits again."""
    from oracle import conv
    M, B, D, L = 2, 3, 16, 1500
    w = datagen.Workload("ddfix", M, B, D, L, decay=300.0, seed=4)
    say(f"[dd fixed filter] M={M} B={B} D={D} L={L}")
    h = torch.from_numpy(datagen.filters_np(w)).to(dev())            # [M, D, L]
    rho = h.permute(2, 0, 1)[:, :, None, :].expand(L, M, B, D).contiguous()
    y = datagen.y_torch(w, dev())
    ctx = _ctx(w, "default")
    z1 = _run(ctx, y, rho)
    ctx.reset()
    assert ctx.position == 0
    z2 = _run(ctx, y, rho)
    assert np.array_equal(z1, z2)
    zr = conv.causal_conv_fft(y.cpu().numpy().reshape(L, -1).astype(np.float64),
                              rho.cpu().numpy().reshape(L, -1).astype(np.float64))
    assert rel_err(z1.reshape(L, -1), zr) <= TOL


def test_dd_errors():
    lcsm = lcsm_mod()
    w = datagen.Workload("dderr", 1, 1, 8, 40, decay=10.0, seed=2)
    ctx = _ctx(w, "default")
    y, rho = datagen.y_torch(w, dev()), datagen.rho_torch(w, dev())
    with pytest.raises(ValueError):
        ctx.step(y[0], rho[0][..., :1])
    _run(ctx, y, rho)
    with pytest.raises(lcsm.LcsmError) as ex:
        ctx.step(y[0], rho[0])
    assert ex.value.code == lcsm.LCSM_EDONE


@pytest.mark.parametrize("name", ["m1b8d768l8k", "m32b16d2048l16k", "m18b4d768l32k",
                                  "m18b1d1024l128k"])
def test_dd_workload_sizes_sampled_columns(name):
    """Full-width contexts with default options: the bench workload (largest
    tile 2U = 4096), L = 16384 (2U = 8192, the largest single-pass tile), and
    L = 32768 and 131072, whose tiles of U = 8192 .. 32768 run as 2x2 .. 8x8
    pairs of 4096-row blocks.  The columns are independent, so sampled ones
    are checked over all L positions: against the definition up to 16384
    positions, beyond that against the oracle's whole-sequence fp64 FFT
    convolution (z is the causal convolution of y and rho)."""
    from oracle import conv
    from oracle.dd import product_naive
    w = datagen.WORKLOADS[name]
    say(f"[dd workload] {name} M={w.M} B={w.B} D={w.D} L={w.L}")
    ctx = lcsm_mod().Dd(w.M, w.B, w.D, w.L)
    cols = datagen.sample_columns(w, 8, seed=91)
    cm, cb, cd = (torch.as_tensor(cols[:, k], device=dev()) for k in range(3))
    chunk = 256 if w.M * w.B * w.D <= (1 << 17) else 32
    z = torch.empty((chunk, w.M, w.B, w.D), dtype=torch.float32, device=dev())
    got, ys, rs = [], [], []
    for t0 in range(0, w.L, chunk):
        t1 = min(w.L, t0 + chunk)
        y = datagen.y_torch(w, dev(), t0, t1)
        rho = datagen.rho_torch(w, dev(), t0, t1)
        for k in range(t1 - t0):
            ctx.step(y[k], rho[k], z[k])
        got.append(z[: t1 - t0, cm, cb, cd].cpu())
        ys.append(y[:, cm, cb, cd].cpu())
        rs.append(rho[:, cm, cb, cd].cpu())
        if t0 % 16384 == 0 and t0:
            say(f"  position {t0}")
    torch.cuda.synchronize()
    ctx.close()
    zg = torch.cat(got).numpy()
    yc, rc = torch.cat(ys).numpy(), torch.cat(rs).numpy()
    if w.L <= 16384:
        zr = product_naive(yc, rc)
    else:
        zr = conv.causal_conv_fft(yc.astype(np.float64), rc.astype(np.float64))
    err = rel_err(zg, zr)
    say(f"  sampled rel err {err:.3e}")
    assert err <= TOL
