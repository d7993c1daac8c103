"""GPU parity of the lazy and eager online convolutions (the baselines of
Sec. 3.1.1, parallel across layers and per layer) against the oracle, through
the C ABI of include/lcsm_base.h (needs an MI355X).

Bars: bit-exact on small-integer data (every partial sum is an integer below
2^24, exact in fp32); max|z_gpu - z_ref| <= 1e-4 max|z_ref| against the fp64
lazy loop on random data; the parallel and the per-layer variant of a kind
run the same kernels on the same sums, so they agree bit for bit."""
import numpy as np
import pytest
import torch

import datagen
from oracle import conv

from gpu_harness import TOL, dev, lcsm_mod, rel_err, say

pytestmark = pytest.mark.gpu

KINDS = ["lazy", "lazy_np", "eager", "eager_np"]
# the last two run the lazy step as partial sums + reduction (t > 256) and
# the eager step over several row chunks per launch
SHAPES = [(2, 3, 40, 300), (3, 1, 5, 1), (1, 1, 1, 77), (1, 2, 64, 600), (2, 2, 300, 700)]


def _run(kind, h, y, B):
    lcsm = lcsm_mod()
    L = y.shape[0]
    ctx = lcsm.Base(kind, torch.from_numpy(h).to(dev()), B)
    yd = torch.from_numpy(np.ascontiguousarray(y)).to(dev())
    z = torch.empty_like(yd)
    for t in range(L):
        ctx.step(yd[t], z[t])
    torch.cuda.synchronize()
    assert ctx.position == L
    out = z.cpu().numpy()
    ctx.close()
    return out


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("kind", KINDS)
def test_integer_data_bit_exact(shape, kind):
    M, B, D, L = shape
    say(f"[base int-exact] {kind} M={M} B={B} D={D} L={L}")
    w = datagen.Workload("bint", M, B, D, L, decay=1.0, seed=sum(shape) + 3)
    h = datagen.int_filters_np(w, 3)
    y = datagen.int_y_np(w, 3)
    z = _run(kind, h, y, B)
    hi, yi = h.astype(np.int64), y.astype(np.int64)
    for m in range(M):
        for b in range(B):
            for d in range(D):
                want = np.convolve(yi[:, m, b, d], hi[m, d])[:L]
                assert np.array_equal(z[:, m, b, d].astype(np.int64), want), (m, b, d)


@pytest.mark.parametrize("shape", [(2, 3, 40, 300), (1, 2, 64, 600)])
@pytest.mark.parametrize("kind", KINDS)
def test_random_data_against_lazy_oracle(shape, kind):
    M, B, D, L = shape
    say(f"[base random] {kind} M={M} B={B} D={D} L={L}")
    w = datagen.Workload("brand", M, B, D, L, decay=L / 3, seed=17)
    h = datagen.filters_np(w)
    y = datagen.y_np(w)
    z = _run(kind, h, y, B)
    # columns [L, n] for the oracle's lazy loop
    yc = y.reshape(L, -1).astype(np.float64)
    hc = np.broadcast_to(h.transpose(2, 0, 1)[:, :, None, :], (L, M, B, D)).reshape(L, -1)
    zr = conv.causal_conv_naive(yc, hc.astype(np.float64))
    err = rel_err(z.reshape(L, -1), zr)
    say(f"  rel err {err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("kind", ["lazy", "eager"])
def test_parallel_equals_per_layer(kind):
    M, B, D, L = 3, 2, 70, 520
    say(f"[base parallel vs per-layer] {kind} M={M} B={B} D={D} L={L}")
    w = datagen.Workload("bnp", M, B, D, L, decay=100.0, seed=5)
    h = datagen.filters_np(w)
    y = datagen.y_np(w)
    assert np.array_equal(_run(kind, h, y, B), _run(kind + "_np", h, y, B))


def test_reset_and_done():
    lcsm = lcsm_mod()
    M, B, D, L = 1, 2, 8, 20
    w = datagen.Workload("bres", M, B, D, L, decay=4.0, seed=9)
    h = torch.from_numpy(datagen.filters_np(w)).to(dev())
    y = torch.from_numpy(datagen.y_np(w)).to(dev())
    for kind in ("lazy", "eager"):
        ctx = lcsm.Base(kind, h, B)
        z1 = torch.empty_like(y)
        for t in range(L):
            ctx.step(y[t], z1[t])
        with pytest.raises(lcsm.LcsmError) as e:
            ctx.step(y[0])
        assert e.value.code == lcsm.LCSM_EDONE
        ctx.reset()
        assert ctx.position == 0
        z2 = torch.empty_like(y)
        for t in range(L):
            ctx.step(y[t], z2[t])
        torch.cuda.synchronize()
        assert torch.equal(z1, z2)
        ctx.close()
