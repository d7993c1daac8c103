"""Tile order of the relaxed online convolution (test infrastructure).

Alg. 1 ("Fast Relaxed Polynomial Interpolation"), 1-indexed: at iteration
i = 1..L-1 the side U is the largest power of two dividing i; the red cell adds
y_i rho_0 into z_i, and the gray tile adds the contribution of y_[i-U+1, i] to
z_[i+1, i+U].  After the loop a final red cell completes z_L.

0-indexed (positions 0..L-1, the convention used throughout this code base):
after z_t has been emitted at step t, the gray tile with i = t + 1 (when
i < L) takes the inputs y[i-U, i) to the outputs z[i, i+U) using the filter
lags 1..2U-1.  When L is not a power of two the output window is clipped at L
(the paper rounds L up instead, Sec. 3 opening).
"""
from __future__ import annotations


def lowbit(i: int) -> int:
    """Largest power of two dividing i (i >= 1)."""
    if i < 1:
        raise ValueError("lowbit needs i >= 1")
    u = 1
    while i % (2 * u) == 0:
        u *= 2
    return u


def tile_after_step(t: int, L: int):
    """The gray tile run after z_t is emitted, or None after the last step.

    Returns (i, U, src_lo, src_hi, dst_lo, dst_hi): inputs y[src_lo, src_hi),
    outputs z[dst_lo, dst_hi).
    """
    if not 0 <= t < L:
        raise ValueError("step out of range")
    i = t + 1
    if i >= L:
        return None
    U = lowbit(i)
    return (i, U, i - U, i, i, min(i + U, L))


def all_tiles(L: int):
    """Every gray tile of a length-L run, in execution order."""
    out = []
    for t in range(L):
        tile = tile_after_step(t, L)
        if tile is not None:
            out.append(tile)
    return out
