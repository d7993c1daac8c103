"""Shared helpers of the GPU tests: drive the library through its binding on
seeded inputs, bring back sampled columns, and compute the oracle's answer for
exactly those columns on the CPU."""
from __future__ import annotations

import sys

import numpy as np
import torch

import datagen
from oracle import conv

TOL = 1e-4  # max|z_gpu - z_ref| <= TOL * max|z_ref|


def say(*args):
    """Progress line naming the case, flushed before GPU work starts."""
    print(*args, flush=True)
    sys.stdout.flush()


def dev():
    return torch.device("cuda:0")


def lcsm_mod():
    import paper_2410_12982_amd.lcsm as lcsm
    return lcsm


def make_ctx(w: datagen.Workload, filters=None, options=None):
    lcsm = lcsm_mod()
    if filters is None:
        filters = datagen.filters_torch(w, dev())
    return lcsm.Lcsm(filters, w.B, options=options), filters


def run_sampled(ctx, w: datagen.Workload, cols, chunk=256, y_fn=None):
    """Teacher-forced run over all L positions; returns z[t, k] for the sampled
    (m, b, d) columns ``cols`` [n, 3] as a numpy fp32 array [L, n].

    Inputs come from the shared generator chunk by chunk (``y_fn(t0, t1)``
    returns a [t1-t0, M, B, D] CUDA tensor; default datagen.y_torch)."""
    if y_fn is None:
        def y_fn(t0, t1):
            return datagen.y_torch(w, dev(), t0, t1)
    m = torch.as_tensor(cols[:, 0], device=dev())
    b = torch.as_tensor(cols[:, 1], device=dev())
    d = torch.as_tensor(cols[:, 2], device=dev())
    out = []
    zbuf = torch.empty((chunk, w.M, w.B, w.D), dtype=torch.float32, device=dev())
    for t0 in range(0, w.L, chunk):
        t1 = min(w.L, t0 + chunk)
        y = y_fn(t0, t1).contiguous()
        ctx.run(y, zbuf, n=t1 - t0)
        out.append(zbuf[: t1 - t0, m, b, d].cpu())
    torch.cuda.synchronize()
    return torch.cat(out).numpy()


def oracle_sampled(w: datagen.Workload, cols, filters_np_fn=None, y_cols=None):
    """fp64 static-FFT oracle for the sampled columns (teacher-forced inputs
    regenerated on the host by the shared generator)."""
    n = len(cols)
    h = np.empty((w.L, n), dtype=np.float64)
    y = np.empty((w.L, n), dtype=np.float64)
    for k, (m, b, d) in enumerate(cols):
        if filters_np_fn is None:
            h[:, k] = datagen.filters_np(w, m_idx=[m], d_idx=[d])[0, 0]
        else:
            h[:, k] = filters_np_fn(m, d)
        if y_cols is None:
            y[:, k] = datagen.y_np(w, m_idx=[m], b_idx=[b], d_idx=[d])[:, 0, 0, 0]
        else:
            y[:, k] = y_cols[:, k]
    return conv.causal_conv_fft(y, h)


def rel_err(z_gpu, z_ref):
    scale = np.abs(z_ref).max()
    return float(np.abs(z_gpu.astype(np.float64) - z_ref).max() / max(scale, 1e-300))


def say_maxima(z_gpu, z_ref, cols):
    """Log, beside the gated maximum, the error maximum of each layer and the
    worst column (z_* are [L, n] over the sampled columns ``cols`` [n, 3] of
    (m, b, d)), each relative to the config's max|z_ref|."""
    scale = max(float(np.abs(z_ref).max()), 1e-300)
    err = np.abs(z_gpu.astype(np.float64) - z_ref).max(axis=0) / scale
    per_layer = {}
    for k, (m, _, _) in enumerate(np.asarray(cols)):
        per_layer[int(m)] = max(per_layer.get(int(m), 0.0), float(err[k]))
    worst = int(np.argmax(err))
    say("  per-layer max rel err: " + ", ".join(f"m{m}={e:.2e}" for m, e in sorted(per_layer.items())))
    m, b, d = (int(v) for v in np.asarray(cols)[worst])
    say(f"  worst column (m={m}, b={b}, d={d}): {err[worst]:.3e}; median column {np.median(err):.3e}")
