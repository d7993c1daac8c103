"""Relaxed online convolution with data-dependent filters (test infrastructure).

The appendix on data-dependent filters (Alg. 5) treats a filter rho that is
itself revealed online: rho_t becomes known with y_t, so the tile of the
data-independent algorithm, which needs lags up to 2U-1 while only U of them
exist, cannot be used.  Instead the contributions are tiled as in van der
Hoeven's relaxed multiplication, with untruncated convolutions of two
length-U blocks (parallelogram tiles).  0-indexed, per column:

    z_t = sum_{j+k=t} y_j rho_k.

At step t, after z_t is emitted (red cell: z_t = acc_t + y_t rho_0 +
y_0 rho_t, the last term only for t >= 1), with the dyadic blocks
[U, 2U) of positions >= 1:

* for every power of two U dividing t+1 with 2U < t+1 (a "rectangle" pair):
  acc[t+1, t+2U) += y[U,2U) (*) rho[t-U+1, t+1) + rho[U,2U) (*) y[t-U+1, t+1);
* if t+1 = 2U for a power of two U (a "square"):
  acc[2U, 4U-1) += y[U,2U) (*) rho[U,2U);

where (*) is the full (2U-1 outputs) convolution; outputs past L-1 are
dropped.  Reading: Alg. 5 as printed keeps only the largest U dividing t+1,
which leaves pairs uncovered (y_1 rho_3 for one); the text says the tiling
is van der Hoeven's, whose step takes every such U, and with every U each
pair (j, k) is covered exactly once (pinned in tests/test_oracle_dd.py).

fp64 numpy; np.convolve is the library primitive for (*).
"""
from __future__ import annotations

import numpy as np


def dd_tiles_after_step(t: int, L: int):
    """Tiles run after step t, in increasing U: tuples (kind, U, recent_lo,
    dst_lo, dst_hi) with kind "rect" or "square"; the fixed blocks are
    [U, 2U), the recent ones [recent_lo, recent_lo + U); outputs go to
    [dst_lo, dst_hi) (clipped at L; tiles with nothing below L are left out)."""
    i1 = t + 1
    out = []
    U = 1
    while i1 % U == 0 and 2 * U <= i1:
        if i1 == 2 * U:
            kind, lo, d0 = "square", U, 2 * U
        else:
            kind, lo, d0 = "rect", t - U + 1, t + 1
        d1 = min(d0 + 2 * U - 1, L)
        if d0 < L:
            out.append((kind, U, lo, d0, d1))
        U *= 2
    return out


def full_conv(a, b):
    """Untruncated convolution of [U, C] blocks along axis 0 -> [2U-1, C]."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    out = np.zeros((a.shape[0] + b.shape[0] - 1,) + a.shape[1:], dtype=np.float64)
    for c in np.ndindex(a.shape[1:]):
        out[(slice(None),) + c] = np.convolve(a[(slice(None),) + c], b[(slice(None),) + c])
    return out


def relaxed_dd(y, rho):
    """Run the tiling above over all positions: y, rho [L, ...] (rho_t is
    read only at step t and later, like y_t).  Returns z [L, ...] fp64."""
    y = np.asarray(y, dtype=np.float64)
    rho = np.asarray(rho, dtype=np.float64)
    L = y.shape[0]
    acc = np.zeros_like(y)
    z = np.zeros_like(y)
    for t in range(L):
        z[t] = acc[t] + y[t] * rho[0]
        if t > 0:
            z[t] += y[0] * rho[t]
        for kind, U, lo, d0, d1 in dd_tiles_after_step(t, L):
            if kind == "square":
                c = full_conv(y[U:2 * U], rho[U:2 * U])
            else:
                c = full_conv(y[U:2 * U], rho[lo:lo + U]) + full_conv(rho[U:2 * U], y[lo:lo + U])
            acc[d0:d1] += c[: d1 - d0]
    return z


def product_naive(y, rho):
    """The plain definition z_t = sum_{j+k=t} y_j rho_k for t < L."""
    y = np.asarray(y, dtype=np.float64)
    rho = np.asarray(rho, dtype=np.float64)
    L = y.shape[0]
    z = np.zeros_like(y)
    for t in range(L):
        z[t] = np.sum(y[: t + 1] * rho[t::-1], axis=0)
    return z
