"""Closed-loop runs at full length on the GPU (needs an MI355X).

The 8192- and 32768-position workloads are specified online: every input
comes from earlier outputs through the tanh chain (lcsm_step_chain).  An fp32
closed loop on these filters is chaotic (rounding noise passes 1e-4 of
max|z| within about 1.7k positions), so no fp32 implementation can follow an
fp64 closed loop to the end.  What is checked instead, at every position of
sampled (b, d) columns through all layers, is that the GPU's run is a
solution of the workload's equations:

* the inputs the chain implies, computed by the oracle's chain rule in fp64
  from the GPU's own outputs, y^0_t = 0.5 tanh(z^{M-1}_{t-1}) + x^0_t and
  y^m_t = 0.5 tanh(z^{m-1}_t) + x^m_t;
* convolved with the filters by the fp64 static-FFT oracle, give the GPU's
  outputs within max|z_gpu - z_ref| <= 1e-4 max|z_ref|.

Differences between the implied inputs and the ones the GPU consumed are one
fp32 tanh rounding each and do not feed back (every implied input comes from
the GPU's outputs, not from the oracle's).
"""
import numpy as np
import pytest
import torch

import datagen
from oracle import conv, feedback

from gpu_harness import TOL, dev, make_ctx, rel_err, say, say_maxima

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,nbd", [("m1b8d768l8k", 24), ("m18b4d768l32k", 6)])
def test_closed_loop_full_length_is_consistent(name, nbd):
    w = datagen.WORKLOADS[name]
    say(f"[closed loop, full length] {w.name} M={w.M} B={w.B} D={w.D} L={w.L}")
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([77, w.B, w.D])))
    bd = {(0, 0), (w.B - 1, w.D - 1), (0, w.D - 1)}
    while len(bd) < nbd:
        bd.add((int(rng.integers(w.B)), int(rng.integers(w.D))))
    bd = sorted(bd)
    cols = np.array([(m, b, d) for b, d in bd for m in range(w.M)], dtype=np.int64)
    ctx, filters = make_ctx(w)
    del filters
    m_i = torch.as_tensor(cols[:, 0], device=dev())
    b_i = torch.as_tensor(cols[:, 1], device=dev())
    d_i = torch.as_tensor(cols[:, 2], device=dev())
    chunk = 256
    zbuf = torch.empty((chunk, w.M, w.B, w.D), dtype=torch.float32, device=dev())
    out = []
    for t0 in range(0, w.L, chunk):
        t1 = min(w.L, t0 + chunk)
        x = datagen.x_torch(w, dev(), t0, t1)
        for t in range(t0, t1):
            ctx.step_chain(x[t - t0], zbuf[t - t0])
        out.append(zbuf[: t1 - t0, m_i, b_i, d_i].cpu())
    torch.cuda.synchronize()
    ctx.close()
    zg = torch.cat(out).numpy()                          # [L, n], n = nbd * M
    n = len(bd)
    # [L, M, n] views of the GPU outputs and the additive inputs per (b, d)
    z3 = zg.reshape(w.L, n, w.M).transpose(0, 2, 1).astype(np.float64)
    x3 = np.stack([datagen.x_np(w, m_idx=np.arange(w.M), b_idx=[b], d_idx=[d])[:, :, 0, 0]
                   for b, d in bd], axis=2)              # [L, M, n]
    rule = feedback.tanh_chain(x3, w.M)
    y3 = np.empty_like(z3)
    for t in range(w.L):
        prev = z3[t - 1] if t else None
        for m in range(w.M):
            y3[t, m] = rule(t, m, z3[t], prev)
    h = np.stack([datagen.filters_np(w, m_idx=[m], d_idx=[d])[0, 0] for m, b, d in cols],
                 axis=1).astype(np.float64)              # [L, n*M] in cols order
    y_cols = y3.transpose(0, 2, 1).reshape(w.L, n * w.M)
    zr = conv.causal_conv_fft(y_cols, h)
    err = rel_err(zg, zr)
    say(f"  rel err {err:.3e} over {len(cols)} columns x {w.L} positions (max|z| {np.abs(zr).max():.3g})")
    say_maxima(zg, zr, cols)
    assert np.isfinite(zg).all()
    assert err <= TOL
