"""The relaxed (tiled) online convolution and the lazy online loop (test infrastructure).

Columns are laid out as [M, C]: M layers, C independent (batch row, channel)
columns per layer, each with its own filter.  Filters are given time-first as
``h[k, m, c]`` (lag k = 0..L-1).  Arithmetic is fp64.
"""
from __future__ import annotations

import numpy as np

from .schedule import tile_after_step


def tau_direct(y_blk, h, U):
    """Contribution of a block of U inputs to the next U outputs (Eq. taus).

    ``y_blk[k]`` = y[i-U+k] for k < U; returns out[j] = sum_k y_blk[k] h[U+j-k]
    for j < U, i.e. the tile y[i-U, i) -> z[i, i+U), which uses lags 1..2U-1.
    """
    out = np.zeros(y_blk.shape, dtype=np.float64)
    for j in range(U):
        for k in range(U):
            out[j] += y_blk[k] * h[U + j - k]
    return out


def tau_fft(y_blk, h, U):
    """The same block via a 2U-point cyclic convolution (Lemma 1, App. B).

    The U inputs are right-padded with U zeros and cyclically convolved with
    the filter prefix h[0, 2U); of the 2U outputs, those at [U, 2U) are the
    wanted ones, untouched by the wrap-around (which lands on [0, U-1)).
    """
    n = 2 * U
    Y = np.fft.rfft(y_blk, n=n, axis=0)
    H = np.fft.rfft(h[:n], n=n, axis=0)
    return np.fft.irfft(Y * H, n=n, axis=0)[U:n]


def tau_direct_vec(y_blk, h, U):
    """tau_direct with the inner sum over k vectorised (same arithmetic order
    is not guaranteed; exact on integer data)."""
    out = np.empty(y_blk.shape, dtype=np.float64)
    for j in range(U):
        # lags U+j-k for k = 0..U-1 are h[j+1 .. U+j] read backwards
        out[j] = np.sum(y_blk * h[j + 1:U + j + 1][::-1], axis=0)
    return out


TAUS = {"direct": tau_direct, "direct_vec": tau_direct_vec, "fft": tau_fft}


class RelaxedOnline:
    """State of Alg. 3 (Alg. 1 run for every layer and column, gray tiles of
    all layers together after the red cells of a position).

    ``acc[t]`` holds, for positions t not yet emitted, the sum of the
    contributions already accounted for; ``y[t]`` the inputs seen so far.
    """

    def __init__(self, h, tau="auto", fft_min_U=32):
        self.h = np.asarray(h, dtype=np.float64)          # [L, M, C]
        self.L = self.h.shape[0]
        self.acc = np.zeros(self.h.shape, dtype=np.float64)
        self.y = np.zeros(self.h.shape, dtype=np.float64)
        self.t = 0
        self.tau = tau
        self.fft_min_U = fft_min_U
        self.tiles = []                                    # executed tiles, for tests

    def _tau(self, U):
        if self.tau == "auto":
            return tau_fft if U >= self.fft_min_U else tau_direct_vec
        return TAUS[self.tau]

    def red(self, m, y_m):
        """Red cell of layer m at the current position: z = acc + y * h_0."""
        t = self.t
        self.y[t, m] = y_m
        return self.acc[t, m] + y_m * self.h[0, m]

    def gray(self):
        """Gray tiles of all layers for i = t + 1, then advance the position."""
        tile = tile_after_step(self.t, self.L)
        if tile is not None:
            i, U, s0, s1, d0, d1 = tile
            tau = self._tau(U)
            # the filter needs lags up to 2U-1; positions past L-1 are never
            # used for outputs kept (d1 <= L), pad with zeros for the window
            hseg = self.h[: 2 * U]
            if hseg.shape[0] < 2 * U:
                pad = np.zeros((2 * U - hseg.shape[0],) + hseg.shape[1:])
                hseg = np.concatenate([hseg, pad], axis=0)
            contrib = tau(self.y[s0:s1], hseg, U)
            self.acc[d0:d1] += contrib[: d1 - d0]
            self.tiles.append(tile)
        self.t += 1


def relaxed_online(h, rule, tau="auto", fft_min_U=32):
    """Run Alg. 3 over all L positions with the input rule ``rule``.

    h: [L, M, C] filters.  Returns (z, y), both [L, M, C] fp64.
    """
    st = RelaxedOnline(h, tau=tau, fft_min_U=fft_min_U)
    L, M, C = st.h.shape
    z = np.zeros((L, M, C), dtype=np.float64)
    for t in range(L):
        for m in range(M):
            y_m = rule(t, m, z[t], z[t - 1] if t > 0 else None)
            z[t, m] = st.red(m, y_m)
        st.gray()
    return z, st.y


def lazy_online(h, rule):
    """The lazy approach (Sec. 3.1.1) driven by the same input rule.

    At each position the output is the direct sum over all inputs so far.
    h: [L, M, C].  Returns (z, y), both [L, M, C] fp64.
    """
    h = np.asarray(h, dtype=np.float64)
    L, M, C = h.shape
    y = np.zeros((L, M, C), dtype=np.float64)
    z = np.zeros((L, M, C), dtype=np.float64)
    for t in range(L):
        for m in range(M):
            y[t, m] = rule(t, m, z[t], z[t - 1] if t > 0 else None)
            z[t, m] = np.sum(y[: t + 1, m] * h[t::-1, m], axis=0)
    return z, y


def filters_to_columns(h_mdl, B):
    """ABI filters h[m, d, k] -> per-column time-first filters [L, M, B*D].

    Column c = b*D + d of layer m uses filter h[m, d, :].
    """
    h_mdl = np.asarray(h_mdl, dtype=np.float64)
    M, D, L = h_mdl.shape
    hc = np.broadcast_to(np.transpose(h_mdl, (2, 0, 1))[:, :, None, :], (L, M, B, D))
    return np.ascontiguousarray(hc.reshape(L, M, B * D))
