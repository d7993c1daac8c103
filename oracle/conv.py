"""Plain definitions of the causal long convolution (test infrastructure).

All functions take the time axis first and broadcast over the remaining
(column) axes.  Arithmetic is fp64.
"""
from __future__ import annotations

import numpy as np


def causal_conv_naive(y, h):
    """Lazy O(L^2) evaluation of Eq. onlineConv, 0-indexed.

    z[t] = sum_{s=0}^{t} y[s] * h[t-s] for every column; y and h are [L, ...]
    with broadcastable column axes.  This is the "lazy approach" of
    Sec. 3.1.1: each output is the formula applied directly.
    """
    y = np.asarray(y, dtype=np.float64)
    h = np.asarray(h, dtype=np.float64)
    L = y.shape[0]
    shape = np.broadcast_shapes(y.shape[1:], h.shape[1:])
    z = np.zeros((L,) + shape, dtype=np.float64)
    for t in range(L):
        # y[0..t] against h[t..0]
        z[t] = np.sum(y[: t + 1] * h[t::-1], axis=0)
    return z


def causal_conv_fft(y, h):
    """Static (whole-sequence) FFT evaluation of the same sum.

    This is how the convolution is computed when all of y is known in advance
    (Sec. 2.3.1, "The Inference Problem"): a linear convolution via a
    zero-padded transform of length >= 2L, truncated to the first L outputs.
    """
    y = np.asarray(y, dtype=np.float64)
    h = np.asarray(h, dtype=np.float64)
    L = y.shape[0]
    n = 1
    while n < 2 * L:
        n *= 2
    Y = np.fft.rfft(y, n=n, axis=0)
    H = np.fft.rfft(h, n=n, axis=0)
    return np.fft.irfft(Y * H, n=n, axis=0)[:L]


def geometric_recurrence(y, r):
    """Output of the convolution with the geometric filter h_k = r^k.

    The filter is the impulse response of a one-state LTI system
    (u_t = r u_{t-1} + y_t, z_t = u_t; rho_i = C^T A^i B with A = r, B = C = 1,
    App. "State Space Models"), so z_t = r z_{t-1} + y_t with z_{-1} = 0.
    """
    y = np.asarray(y, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    z = np.zeros(np.broadcast_shapes(y.shape, (1,) + r.shape), dtype=np.float64)
    prev = np.zeros(z.shape[1:], dtype=np.float64)
    for t in range(y.shape[0]):
        prev = r * prev + y[t]
        z[t] = prev
    return z
