"""Seeded synthetic inputs for the relaxed online long convolution.

This module is shared by the CPU oracle and by the GPU tests/bench. It holds
no arithmetic of the convolution method itself: only a counter-based random
generator and the workload shapes.

Generator (counter-based, so any subset of elements can be drawn on its own):

* ``hash32`` is the "lowbias32" integer hash (C. Wellons, 2018):
  ``x ^= x>>16; x *= 0x7feb352d; x ^= x>>15; x *= 0x846ca68b; x ^= x>>16``
  on 32-bit words.
* Element ``n`` (a flat index of a tensor) of draw ``j`` of stream ``s`` under
  seed ``seed`` gets the 32-bit word
  ``hash32(hash32(lo ^ k) ^ hi ^ k2)`` with ``lo, hi`` the low/high 32 bits
  of ``n``, ``k = hash32((seed*0x9E3779B1 + s*0x85EBCA77 + j*0xC2B2AE3D) mod
  2^32)`` and ``k2 = hash32((k + 1) mod 2^32)``.  For a fixed ``hi`` the map
  ``lo -> word`` is a bijection, so no two elements of a tensor below 2^32
  elements share a word.
* ``uniform`` keeps the top 24 bits: ``u = (w >> 8) / 2^24`` in [0, 1), exact
  in fp32.
* ``normal`` is the Irwin-Hall(4) stand-in for N(0,1):
  ``g = (u_0+u_1+u_2+u_3 - 2) * sqrt(3)`` evaluated in fp64 (the sum is exact,
  the product is one IEEE rounding), so numpy and torch agree bit for bit.

The word functions accept numpy arrays (uint64 words) or torch tensors (int64
words, any device) and return the same kind.  Multiplication mod 2^32 is split
into 16-bit halves so that no intermediate overflows 63 bits on either one.

Tensors and their flat index order:

* filters ``h[m, d, k]`` (the ABI layout [M][D][L]):  ``n = (m*D + d)*L + k``,
  stream 0.  ``h = fp32(g * exp(-k/decay))``, the decay table is evaluated
  once in fp64 by numpy and shared by both backends.
* teacher-forced inputs ``y[t, m, b, d]``: ``n = ((t*M + m)*B + b)*D + d``,
  stream 1, ``y = u - 1/2`` (uniform on [-1/2, 1/2), exact in fp32).
* additive chain inputs ``x[t, m, b, d]``: same index, stream 2,
  ``x = fp32(sigma * g)``.
* small-integer data (bit-exact tests): ``v = (w mod (2r+1)) - r``.
* weights of the synthetic model's MLP blocks (the [out][in] layout):
  ``w_up[m, n, k]`` (n < 2D, k < D, index ``(m*2D + n)*D + k``, stream 3),
  ``b_up[m, n]`` (``m*2D + n``, stream 4), ``w_down[m, n, k]`` (n < D,
  k < 2D, ``(m*D + n)*2D + k``, stream 5), ``b_down[m, n]`` (``m*D + n``,
  stream 6).  ``w_up = fp32(g / sqrt(D))``, ``w_down = fp32(g * s / sqrt(2D))``
  with ``s = 1 / (2 * sqrt(sum_k exp(-2k/decay)))`` (the inverse of twice a
  filter's expected L2 norm, so that a layer -- mixer then block -- does not
  amplify and the closed loop stays bounded), biases ``fp32(0.1 g)``.
* sampler noise ``eps[t, b, d]``: ``n = (t*B + b)*D + d``, stream 7,
  ``eps = fp32(sigma * g)``.
* data-dependent filter inputs ``rho[t, m, b, d]`` (revealed with y_t):
  index as y, stream 8, ``rho = fp32(g * exp(-t/decay))`` (a filter's
  decaying profile, drawn per batch row as well).
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

M32 = 0xFFFFFFFF

# stream ids
FILTERS, YIN, XIN = 0, 1, 2
W_UP, B_UP, W_DOWN, B_DOWN, NOISE = 3, 4, 5, 6, 7
RHO = 8


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: M layers, B batch rows, D channels, L positions.

    ``decay`` is the filter decay length (h[k] ~ N(0,1) * exp(-k/decay)),
    ``x_sigma`` the standard deviation of the additive chain input x.
    """
    name: str
    M: int
    B: int
    D: int
    L: int
    decay: float
    x_sigma: float = 0.1
    seed: int = 0

    @property
    def columns(self) -> int:
        return self.M * self.B * self.D


# The five workloads: shapes and filter decays as stated for the benchmark.
WORKLOADS = {
    w.name: w
    for w in [
        Workload("m1b1d16l1k", 1, 1, 16, 1024, decay=200.0, seed=1),
        Workload("m1b8d768l8k", 1, 8, 768, 8192, decay=2048.0, seed=2),
        Workload("m18b4d768l32k", 18, 4, 768, 32768, decay=2048.0, seed=3),
        Workload("m18b1d1024l128k", 18, 1, 1024, 131072, decay=16384.0, seed=4),
        Workload("m32b16d2048l16k", 32, 16, 2048, 16384, decay=2048.0, seed=5),
    ]
}


def _is_torch(a) -> bool:
    return type(a).__module__.startswith("torch")


def _mul32(x, c: int):
    """(x * c) mod 2^32 for word arrays x < 2^32, without 64-bit overflow."""
    lo = (x & 0xFFFF) * c
    hi = (((x >> 16) * (c & 0xFFFF)) & 0xFFFF) << 16
    return (lo + hi) & M32


def hash32(x):
    """lowbias32 on an integer array of 32-bit words (numpy uint64 / torch int64)."""
    x = x & M32
    x = x ^ (x >> 16)
    x = _mul32(x, 0x7FEB352D)
    x = x ^ (x >> 15)
    x = _mul32(x, 0x846CA68B)
    x = x ^ (x >> 16)
    return x


def _hash32_int(x: int) -> int:
    x &= M32
    x ^= x >> 16
    x = (x * 0x7FEB352D) & M32
    x ^= x >> 15
    x = (x * 0x846CA68B) & M32
    x ^= x >> 16
    return x


def _key(seed: int, stream: int, draw: int) -> int:
    return _hash32_int((seed * 0x9E3779B1 + stream * 0x85EBCA77 + draw * 0xC2B2AE3D) & M32)


def words(n, seed: int, stream: int, draw: int = 0):
    """32-bit random words for flat indices ``n`` (numpy uint64 or torch int64 array)."""
    k = _key(seed, stream, draw)
    k2 = _hash32_int(k + 1)
    lo = n & M32
    hi = n >> 32
    return hash32(hash32(lo ^ k) ^ hi ^ k2)


def _as_index(n, like=None):
    if _is_torch(n):
        import torch
        return n.to(torch.int64)
    return np.asarray(n, dtype=np.uint64)


def uniform(n, seed: int, stream: int, draw: int = 0):
    """Uniform [0,1) with 24-bit resolution, returned as fp64 (exact)."""
    n = _as_index(n)
    w = words(n, seed, stream, draw) >> 8
    if _is_torch(w):
        import torch
        return w.to(torch.float64) * (2.0 ** -24)
    return w.astype(np.float64) * (2.0 ** -24)


def normal(n, seed: int, stream: int):
    """Irwin-Hall(4) approximately-N(0,1) draws in fp64 (exact sum, one rounding)."""
    s = uniform(n, seed, stream, 0)
    for j in range(1, 4):
        s = s + uniform(n, seed, stream, j)
    return (s - 2.0) * math.sqrt(3.0)


def small_int(n, seed: int, stream: int, r: int):
    """Integers in [-r, r] as fp64."""
    n = _as_index(n)
    w = words(n, seed, stream, 7)
    v = w % (2 * r + 1)
    if _is_torch(v):
        import torch
        return v.to(torch.float64) - r
    return v.astype(np.float64) - r


def decay_table(L: int, decay: float) -> np.ndarray:
    """exp(-k/decay) for k < L, fp64 (numpy)."""
    return np.exp(-np.arange(L, dtype=np.float64) / decay)


# ---------------------------------------------------------------- numpy views

def filters_np(w: Workload, m_idx=None, d_idx=None, lags=None) -> np.ndarray:
    """Filters h[m, d, k] as fp32 numpy, for the selected layers/channels and
    the first ``lags`` lags (default all L).

    Returns shape [len(m_idx), len(d_idx), lags].
    """
    m_idx = np.arange(w.M) if m_idx is None else np.asarray(m_idx)
    d_idx = np.arange(w.D) if d_idx is None else np.asarray(d_idx)
    lags = w.L if lags is None else lags
    k = np.arange(lags, dtype=np.uint64)
    n = ((m_idx[:, None, None].astype(np.uint64) * np.uint64(w.D)
          + d_idx[None, :, None].astype(np.uint64)) * np.uint64(w.L) + k[None, None, :])
    g = normal(n, w.seed, FILTERS)
    return (g * decay_table(w.L, w.decay)[None, None, :lags]).astype(np.float32)


def _tmbd_index(w: Workload, t_idx, m_idx, b_idx, d_idx):
    t = np.asarray(t_idx).astype(np.uint64)[:, None, None, None]
    m = np.asarray(m_idx).astype(np.uint64)[None, :, None, None]
    b = np.asarray(b_idx).astype(np.uint64)[None, None, :, None]
    d = np.asarray(d_idx).astype(np.uint64)[None, None, None, :]
    M, B, D = np.uint64(w.M), np.uint64(w.B), np.uint64(w.D)
    return ((t * M + m) * B + b) * D + d


def _sel(w, t_idx, m_idx, b_idx, d_idx):
    return (np.arange(w.L) if t_idx is None else t_idx,
            np.arange(w.M) if m_idx is None else m_idx,
            np.arange(w.B) if b_idx is None else b_idx,
            np.arange(w.D) if d_idx is None else d_idx)


def y_np(w: Workload, t_idx=None, m_idx=None, b_idx=None, d_idx=None) -> np.ndarray:
    """Teacher-forced inputs y[t, m, b, d] (fp32), uniform on [-1/2, 1/2)."""
    n = _tmbd_index(w, *_sel(w, t_idx, m_idx, b_idx, d_idx))
    return (uniform(n, w.seed, YIN) - 0.5).astype(np.float32)


def x_np(w: Workload, t_idx=None, m_idx=None, b_idx=None, d_idx=None) -> np.ndarray:
    """Additive chain inputs x[t, m, b, d] (fp32), sigma * N(0,1) stand-in."""
    n = _tmbd_index(w, *_sel(w, t_idx, m_idx, b_idx, d_idx))
    return (w.x_sigma * normal(n, w.seed, XIN)).astype(np.float32)


def rho_np(w: Workload, t_idx=None, m_idx=None, b_idx=None, d_idx=None) -> np.ndarray:
    """Data-dependent filter inputs rho[t, m, b, d] (fp32), N(0,1) * exp(-t/decay)."""
    sel = _sel(w, t_idx, m_idx, b_idx, d_idx)
    n = _tmbd_index(w, *sel)
    dec = decay_table(w.L, w.decay)[np.asarray(sel[0])][:, None, None, None]
    return (normal(n, w.seed, RHO) * dec).astype(np.float32)


def int_rho_np(w: Workload, r: int = 3) -> np.ndarray:
    """Small-integer data-dependent filter inputs rho[t, m, b, d] in [-r, r] (fp32)."""
    n = np.arange(w.L * w.M * w.B * w.D, dtype=np.uint64)
    return small_int(n, w.seed, RHO, r).reshape(w.L, w.M, w.B, w.D).astype(np.float32)


def int_filters_np(w: Workload, r: int = 3) -> np.ndarray:
    """Small-integer filters h[m, d, k] in [-r, r] (fp32)."""
    n = np.arange(w.M * w.D * w.L, dtype=np.uint64)
    return small_int(n, w.seed, FILTERS, r).reshape(w.M, w.D, w.L).astype(np.float32)


def int_y_np(w: Workload, r: int = 3) -> np.ndarray:
    """Small-integer teacher-forced inputs y[t, m, b, d] in [-r, r] (fp32)."""
    n = np.arange(w.L * w.M * w.B * w.D, dtype=np.uint64)
    return small_int(n, w.seed, YIN, r).reshape(w.L, w.M, w.B, w.D).astype(np.float32)


def mlp_scales(w: Workload):
    """(scale of w_up, scale of w_down, scale of the biases), fp64."""
    norm = math.sqrt(float(np.sum(decay_table(w.L, w.decay) ** 2)))
    return 1.0 / math.sqrt(w.D), 1.0 / (2.0 * norm * math.sqrt(2 * w.D)), 0.1


def _mlp_index_shapes(w: Workload):
    D2 = 2 * w.D
    return ((W_UP, (w.M, D2, w.D), 0), (B_UP, (w.M, D2), 2), (W_DOWN, (w.M, w.D, D2), 1),
            (B_DOWN, (w.M, w.D), 2))


def mlp_weights_np(w: Workload):
    """(w_up [M,2D,D], b_up [M,2D], w_down [M,D,2D], b_down [M,D]) fp32 numpy."""
    sc = mlp_scales(w)
    out = []
    for stream, shape, which in _mlp_index_shapes(w):
        n = np.arange(int(np.prod(shape)), dtype=np.uint64)
        out.append((sc[which] * normal(n, w.seed, stream)).astype(np.float32).reshape(shape))
    return tuple(out)


def noise_np(w: Workload, t0: int = 0, t1: int | None = None) -> np.ndarray:
    """Sampler noise eps[t0:t1, b, d] (fp32)."""
    t1 = w.L if t1 is None else t1
    slab = w.B * w.D
    n = (np.arange(t0, t1, dtype=np.uint64)[:, None] * np.uint64(slab)
         + np.arange(slab, dtype=np.uint64)[None, :])
    return (w.x_sigma * normal(n, w.seed, NOISE)).astype(np.float32).reshape(t1 - t0, w.B, w.D)


# ---------------------------------------------------------------- torch views

def mlp_weights_torch(w: Workload, device):
    """The weights of :func:`mlp_weights_np` as fp32 torch tensors (bit-identical)."""
    import torch
    sc = mlp_scales(w)
    out = []
    for stream, shape, which in _mlp_index_shapes(w):
        total = int(np.prod(shape))
        t = torch.empty(total, dtype=torch.float32, device=device)
        step = 1 << 24
        for a in range(0, total, step):
            n = torch.arange(a, min(total, a + step), device=device, dtype=torch.int64)
            t[a:a + len(n)] = (sc[which] * normal(n, w.seed, stream)).to(torch.float32)
        out.append(t.view(shape))
    return tuple(out)


def noise_torch(w: Workload, device, t0: int = 0, t1: int | None = None):
    """Sampler noise eps[t0:t1, b, d] as an fp32 torch tensor on ``device``."""
    import torch
    t1 = w.L if t1 is None else t1
    slab = w.B * w.D
    out = torch.empty((t1 - t0, w.B, w.D), dtype=torch.float32, device=device)
    flat = out.view(t1 - t0, slab)
    j = torch.arange(slab, device=device, dtype=torch.int64)
    step = max(1, (1 << 22) // slab)
    for a in range(t0, t1, step):
        b = min(t1, a + step)
        ts = torch.arange(a, b, device=device, dtype=torch.int64)
        n = ts[:, None] * slab + j[None, :]
        flat[a - t0:b - t0] = (w.x_sigma * normal(n, w.seed, NOISE)).to(torch.float32)
    return out


def filters_torch(w: Workload, device, m_chunk: int = 1):
    """Filters h[m, d, k] as an fp32 torch tensor [M, D, L] on ``device``.

    Bit-identical to :func:`filters_np`; generated a few layers at a time.
    """
    import torch
    out = torch.empty((w.M, w.D, w.L), dtype=torch.float32, device=device)
    dec = torch.from_numpy(decay_table(w.L, w.decay)).to(device)
    k = torch.arange(w.L, device=device, dtype=torch.int64)
    d = torch.arange(w.D, device=device, dtype=torch.int64)
    for m0 in range(0, w.M, m_chunk):
        ms = torch.arange(m0, min(w.M, m0 + m_chunk), device=device, dtype=torch.int64)
        n = (ms[:, None, None] * w.D + d[None, :, None]) * w.L + k[None, None, :]
        g = normal(n, w.seed, FILTERS)
        out[m0:m0 + len(ms)] = (g * dec[None, None, :]).to(torch.float32)
    return out


def y_torch(w: Workload, device, t0: int = 0, t1: int | None = None):
    """Teacher-forced inputs y[t0:t1, m, b, d] as an fp32 torch tensor on ``device``."""
    import torch
    t1 = w.L if t1 is None else t1
    slab = w.M * w.B * w.D
    out = torch.empty((t1 - t0, w.M, w.B, w.D), dtype=torch.float32, device=device)
    flat = out.view(t1 - t0, slab)
    j = torch.arange(slab, device=device, dtype=torch.int64)
    step = max(1, (1 << 24) // slab)
    for a in range(t0, t1, step):
        b = min(t1, a + step)
        ts = torch.arange(a, b, device=device, dtype=torch.int64)
        n = ts[:, None] * slab + j[None, :]
        flat[a - t0:b - t0] = (uniform(n, w.seed, YIN) - 0.5).to(torch.float32)
    return out


def x_torch(w: Workload, device, t0: int = 0, t1: int | None = None):
    """Additive chain inputs x[t0:t1, m, b, d] as an fp32 torch tensor on ``device``."""
    import torch
    t1 = w.L if t1 is None else t1
    slab = w.M * w.B * w.D
    out = torch.empty((t1 - t0, w.M, w.B, w.D), dtype=torch.float32, device=device)
    flat = out.view(t1 - t0, slab)
    j = torch.arange(slab, device=device, dtype=torch.int64)
    step = max(1, (1 << 22) // slab)
    for a in range(t0, t1, step):
        b = min(t1, a + step)
        ts = torch.arange(a, b, device=device, dtype=torch.int64)
        n = ts[:, None] * slab + j[None, :]
        flat[a - t0:b - t0] = (w.x_sigma * normal(n, w.seed, XIN)).to(torch.float32)
    return out


def rho_torch(w: Workload, device, t0: int = 0, t1: int | None = None):
    """Data-dependent filter inputs rho[t0:t1, m, b, d] as an fp32 torch tensor."""
    import torch
    t1 = w.L if t1 is None else t1
    slab = w.M * w.B * w.D
    out = torch.empty((t1 - t0, w.M, w.B, w.D), dtype=torch.float32, device=device)
    flat = out.view(t1 - t0, slab)
    dec = torch.from_numpy(decay_table(w.L, w.decay)).to(device)
    j = torch.arange(slab, device=device, dtype=torch.int64)
    step = max(1, (1 << 22) // slab)
    for a in range(t0, t1, step):
        b = min(t1, a + step)
        ts = torch.arange(a, b, device=device, dtype=torch.int64)
        n = ts[:, None] * slab + j[None, :]
        flat[a - t0:b - t0] = (normal(n, w.seed, RHO) * dec[a:b, None]).to(torch.float32)
    return out


def sample_columns(w: Workload, count: int, seed: int = 12345):
    """A fixed sample of (m, b, d) columns: the batch/channel boundaries of every
    layer plus seeded random picks.  Returns an int array of shape [n, 3]."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, w.M, w.B, w.D])))
    cols = set()
    for m in sorted({0, w.M - 1}):
        for b in sorted({0, w.B - 1}):
            for d in sorted({0, min(63, w.D - 1), min(64, w.D - 1), w.D - 1}):
                cols.add((m, b, d))
    while len(cols) < min(count, w.columns):
        cols.add((int(rng.integers(w.M)), int(rng.integers(w.B)), int(rng.integers(w.D))))
    return np.array(sorted(cols), dtype=np.int64)
