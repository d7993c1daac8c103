// FFT gray tiles on transposed column chunks, for gfx950.
//
// The row-panel tile kernels (lcsm_fft.hip) read and write each state row in
// pieces of WC complex columns, and at 2U >= 2048 LDS leaves room for only
// 16-64 bytes per row, a run width at which HBM delivers a fraction of its
// bandwidth.  Here a chunk of columns of the tile's input rows is first
// transposed into a column-major scratch (64 x 64 tiles through LDS: 256-byte
// runs on both sides), each workgroup then transforms one complex column --
// two real state columns packed as real and imaginary part -- reading and
// writing it as one contiguous run along time, and a second transpose adds
// the outputs into the destination rows (or stores them, for the in-place
// swap of half-state storage).  28U bytes move per column instead of 12U, at
// full run width.  The spectra of these tile sizes are kept channel-major,
// Hc[m][d][k] (k <= U, pre-scaled by 1/2U), so that a workgroup's spectrum
// loads are contiguous as well.
//
// Transform (as in the row-panel tile, Lemma 1 / App. B): with the two real
// columns a, b of a pair, z = y_a + i y_b over [0, U) and zero above,
// Z = DFT_2U(z); P[k] = Z[k] S[k] + conj(Z[2U-k]) D[k] with S = (Ha + Hb)/2,
// D = (Ha - Hb)/2; the outputs U + j of IDFT_2U(P) are the tile's outputs j
// of column a (real part) and b (imaginary part).
#include "lcsm_fft_core.h"
#include "lcsm_internal.h"

namespace lcsm {
namespace {

using fft::cadd;
using fft::cmul;
using fft::conjf2;

constexpr int kTT = 64;        // transpose tile side
constexpr int kTThreads = 256;  // 64 x 4

// X[(g - g0) * ldx + r] = S[m][row0 + r][c] for global columns g = m*BD + c
// in [g0, g0 + ncols) and r < nrows.  lstride: state floats per layer.
__global__ __launch_bounds__(kTThreads) void k_rows_to_cols(const float* __restrict__ S,
                                                            size_t lstride, int BD, int row0,
                                                            int nrows, long long g0, int ncols,
                                                            float* __restrict__ X, int ldx) {
  __shared__ float tile[kTT][kTT + 1];
  const int cb = (int)blockIdx.x * kTT, rb = (int)blockIdx.y * kTT;
  const int tx = (int)threadIdx.x & (kTT - 1), ty = (int)threadIdx.x / kTT;
  const int col = cb + tx;
  if (col < ncols) {
    const long long g = g0 + col;
    const long long m = g / BD;
    const int c = (int)(g - m * BD);
    const float* src = S + (size_t)m * lstride + (size_t)row0 * BD + c;
#pragma unroll
    for (int k = 0; k < kTT / 4; ++k) {
      const int r = rb + ty + 4 * k;
      if (r < nrows) tile[ty + 4 * k][tx] = src[(size_t)r * BD];
    }
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kTT / 4; ++k) {
    const int cc = cb + ty + 4 * k, r = rb + tx;
    if (cc < ncols && r < nrows) X[(size_t)cc * ldx + r] = tile[tx][ty + 4 * k];
  }
}

// S[m][row0 + r][c] += X[(g - g0) * ldx + r] (STORE: =) for r < nrows.
template <bool STORE>
__global__ __launch_bounds__(kTThreads) void k_cols_to_rows(const float* __restrict__ X, int ldx,
                                                            float* __restrict__ S, size_t lstride,
                                                            int BD, int row0, int nrows,
                                                            long long g0, int ncols) {
  __shared__ float tile[kTT][kTT + 1];
  const int cb = (int)blockIdx.x * kTT, rb = (int)blockIdx.y * kTT;
  const int tx = (int)threadIdx.x & (kTT - 1), ty = (int)threadIdx.x / kTT;
#pragma unroll
  for (int k = 0; k < kTT / 4; ++k) {
    const int cc = cb + ty + 4 * k, r = rb + tx;
    if (cc < ncols && r < nrows) tile[ty + 4 * k][tx] = X[(size_t)cc * ldx + r];
  }
  __syncthreads();
  const int col = cb + tx;
  if (col >= ncols) return;
  const long long g = g0 + col;
  const long long m = g / BD;
  const int c = (int)(g - m * BD);
  float* dst = S + (size_t)m * lstride + (size_t)row0 * BD + c;
#pragma unroll
  for (int k = 0; k < kTT / 4; ++k) {
    const int r = rb + ty + 4 * k;
    if (r < nrows) {
      float* p = dst + (size_t)r * BD;
      *p = STORE ? tile[tx][ty + 4 * k] : *p + tile[tx][ty + 4 * k];
    }
  }
}

// The two transposes with 16-byte accesses on both sides, for B*D, the
// column length ldx and the row count multiples of 4 (then every float4 lies
// in one layer's row and is aligned): a wavefront moves four 256-byte row
// segments (or four column runs) per instruction instead of one.  LDS keeps
// 4-byte elements with a pitch of 65: the row-side lanes (4 rows x 16 float4)
// and the column-side lanes (16 x 4 rows of 4 columns) both meet 64 distinct
// banks.
__global__ __launch_bounds__(kTThreads) void k_rows_to_cols4(const float* __restrict__ S,
                                                             size_t lstride, int BD, int row0,
                                                             int nrows, long long g0, int ncols,
                                                             float* __restrict__ X, int ldx) {
  __shared__ float tile[kTT][kTT + 1];
  const int cb = (int)blockIdx.x * kTT, rb = (int)blockIdx.y * kTT;
  const int q4 = (int)threadIdx.x & 15, r16 = (int)threadIdx.x >> 4;
  const int col = cb + 4 * q4;
  if (col < ncols) {
    const long long g = g0 + col;
    const long long m = g / BD;
    const int c = (int)(g - m * BD);
    const float* src = S + (size_t)m * lstride + (size_t)row0 * BD + c;
#pragma unroll
    for (int k = 0; k < kTT / 16; ++k) {
      const int r = r16 + 16 * k;
      if (rb + r < nrows) {
        const float4 v = *reinterpret_cast<const float4*>(src + (size_t)(rb + r) * BD);
        tile[r][4 * q4] = v.x;
        tile[r][4 * q4 + 1] = v.y;
        tile[r][4 * q4 + 2] = v.z;
        tile[r][4 * q4 + 3] = v.w;
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kTT / 16; ++k) {
    const int cc = r16 + 16 * k, r = 4 * q4;
    if (cb + cc < ncols && rb + r < nrows) {
      const float4 v = make_float4(tile[r][cc], tile[r + 1][cc], tile[r + 2][cc], tile[r + 3][cc]);
      *reinterpret_cast<float4*>(X + (size_t)(cb + cc) * ldx + rb + r) = v;
    }
  }
}

template <bool STORE>
__global__ __launch_bounds__(kTThreads) void k_cols_to_rows4(const float* __restrict__ X, int ldx,
                                                             float* __restrict__ S, size_t lstride,
                                                             int BD, int row0, int nrows,
                                                             long long g0, int ncols) {
  __shared__ float tile[kTT][kTT + 1];
  const int cb = (int)blockIdx.x * kTT, rb = (int)blockIdx.y * kTT;
  const int q4 = (int)threadIdx.x & 15, r16 = (int)threadIdx.x >> 4;
#pragma unroll
  for (int k = 0; k < kTT / 16; ++k) {
    const int cc = r16 + 16 * k, r = 4 * q4;
    if (cb + cc < ncols && rb + r < nrows) {
      const float4 v = *reinterpret_cast<const float4*>(X + (size_t)(cb + cc) * ldx + rb + r);
      tile[r][cc] = v.x;
      tile[r + 1][cc] = v.y;
      tile[r + 2][cc] = v.z;
      tile[r + 3][cc] = v.w;
    }
  }
  __syncthreads();
  const int col = cb + 4 * q4;
  if (col >= ncols) return;
  const long long g = g0 + col;
  const long long m = g / BD;
  const int c = (int)(g - m * BD);
  float* dst = S + (size_t)m * lstride + (size_t)row0 * BD + c;
#pragma unroll
  for (int k = 0; k < kTT / 16; ++k) {
    const int r = r16 + 16 * k;
    if (rb + r < nrows) {
      float4* p = reinterpret_cast<float4*>(dst + (size_t)(rb + r) * BD);
      float4 o = make_float4(tile[r][4 * q4], tile[r][4 * q4 + 1], tile[r][4 * q4 + 2],
                             tile[r][4 * q4 + 3]);
      if constexpr (!STORE) {
        const float4 a = *p;
        o = make_float4(a.x + o.x, a.y + o.y, a.z + o.z, a.w + o.w);
      }
      *p = o;
    }
  }
}

// Two-level twiddles in LDS: w_N^f = hi[f >> 6] * lo[f & 63] with
// hi[j] = w_N^{64 j} (N/64 entries) and lo[l] = w_N^l (64 entries), both
// copied from the fp64-derived global table; one complex product per
// twiddle instead of N entries of LDS.
template <int N>
struct TwSplit {
  static constexpr int NH = N / 64;
  static constexpr bool kRow = true;
  const float2* hi;
  const float2* lo;
  template <bool INV, int NN>
  __device__ __forceinline__ float2 get(int e) const {
    const int f = e * (N / NN);
    const float2 w = cmul(hi[f >> 6], lo[f & 63]);
    return INV ? conjf2(w) : w;
  }
  // The twiddles w^{qk}, 0 < q < R, of one butterfly: the powers of two of
  // q from the table, every other q as the product of its highest power of
  // two and the rest (at most three products deep at R = 16): 2 log2 R LDS
  // reads instead of 2 (R - 1).
  template <bool INV, int NN, int R>
  __device__ __forceinline__ void row(int k, float2 (&w)[R]) const {
#pragma unroll
    for (int p = 1; p < R; p *= 2) w[p] = get<INV, NN>(p * k);
#pragma unroll
    for (int q = 3; q < R; ++q) {
      if (q & (q - 1)) {
        int hb = 1;
        while (2 * hb <= q) hb *= 2;
        w[q] = cmul(w[hb], w[q - hb]);
      }
    }
  }
};

// One complex column per workgroup (consecutive threads take consecutive
// time indices: contiguous loads and stores), N/16 threads: one radix-16
// butterfly per thread and pass, at most 128 registers from 2U = 4096 on
// (four waves per SIMD: two workgroups per CU at 4096 and 8192, one of 1024
// threads at 16384, whose data fills most of LDS).  The full twiddle table
// goes to LDS while it is small, the two-level one above that.
template <int N>
struct ColCfg {
  static constexpr int NT = N / 16 < 64 ? 64 : (N / 16 > 1024 ? 1024 : N / 16);
  static constexpr bool TWL = N <= 1024;
  // waves per SIMD the registers must allow
  static constexpr int MINB = N >= 4096 ? 4 : 1;
  // LDS padding: one slot after every 16 elements.  With one column per
  // workgroup the first pass writes at a stride of 16 elements (128 bytes)
  // and the second in runs of 16 a power of two apart: without it all lanes
  // of a wave meet on one bank, with it at most three share one.
  static constexpr int SH = 4;
  static constexpr int SLOTS = N + (N >> SH);
};

// Chunk columns (ca, cb) of the complex column pr, in the order `mode` sets
// (below); cb may lie past the chunk in mode 0.
__device__ __forceinline__ void col_pair(int pr, int mode, int BD, int D, int B, int& ca, int& cb) {
  if (mode == 2) {
    const int half = B / 2, lp = half * D;  // pairs per layer
    const int l = pr / lp, r = pr - l * lp;
    const int d = r / half, bp = r - d * half;
    ca = l * BD + 2 * bp * D + d;
    cb = ca + D;
  } else {
    if (mode == 1) {
      const int ppr = D / 2, lp = B * ppr;
      const int l = pr / lp, r = pr - l * lp;
      const int dp = r / B, b = r - dp * B;
      pr = l * lp + b * ppr + dp;
    }
    ca = 2 * pr;
    cb = ca + 1;
  }
}

// mode: how the complex columns pair the chunk's real columns.
//   2 (the chunk holds whole layers, B even): batch rows 2p and 2p+1 of one
//     channel -- both share its spectrum, the product is P = Z H, and the
//     workgroups of one channel are consecutive (its spectrum stays in L2);
//   1 (whole layers, D even): channels 2q and 2q+1 of one batch row, the
//     workgroups of one channel pair consecutive over the batch rows;
//   0: neighbouring chunk columns.
template <int N>
__global__ __launch_bounds__(ColCfg<N>::NT, ColCfg<N>::MINB) void k_fft_coltile(float* __restrict__ X, int ldx,
                                                               const float2* __restrict__ Hc,
                                                               const float2* __restrict__ tw,
                                                               long long g0, int ncols, int BD,
                                                               int D, int B, int mode) {
  constexpr int NT = ColCfg<N>::NT, U = N / 2;
  // one channel's spectrum loaded into registers before the transform
  constexpr int HU = (U + 1 + NT - 1) / NT;
  constexpr bool PRE = N <= 8192;
  using TW = typename std::conditional<ColCfg<N>::TWL, fft::TwLds<N>, TwSplit<N>>::type;
  constexpr int SH = ColCfg<N>::SH;
  __shared__ float2 buf[ColCfg<N>::SLOTS];
  __shared__ float2 twl[ColCfg<N>::TWL ? N : N / 64 + 64];
  TW twz;
  if constexpr (ColCfg<N>::TWL) {
    fft::load_twiddles<N, NT>(twl, tw);
    twz = TW{twl};
  } else {
    for (int j = (int)threadIdx.x; j < N / 64; j += NT) twl[j] = tw[N + 64 * j];
    for (int l = (int)threadIdx.x; l < 64; l += NT) twl[N / 64 + l] = tw[N + l];
    twz = TW{twl, twl + N / 64};
  }
  int ca, cb;  // chunk columns of the pair (cb may be past the chunk in mode 0)
  col_pair(fft::xcd_logical((int)blockIdx.x, (int)gridDim.x), mode, BD, D, B, ca, cb);
  const bool hasb = cb < ncols;
  float* xa = X + (size_t)ca * ldx;
  float* xb = X + (size_t)(hasb ? cb : ca) * ldx;
  // spectra of the two columns' channels (contiguous along k)
  const long long ga = g0 + ca, gb = g0 + (hasb ? cb : ca);
  const long long ma = ga / BD, mb = gb / BD;
  const int da = (int)(ga - ma * BD) % D, db = (int)(gb - mb * BD) % D;
  const float2* ha = Hc + ((size_t)ma * D + da) * (U + 1);
  const float2* hb = Hc + ((size_t)mb * D + db) * (U + 1);
  float2 hv[PRE ? HU : 1];
  if constexpr (PRE) {
    if (mode == 2) {
#pragma unroll
      for (int j = 0; j < HU; ++j) {
        const int kk = (int)threadIdx.x + j * NT;
        hv[j] = kk <= U ? ha[kk] : make_float2(0.f, 0.f);
      }
    }
  }
  fft::forward_from_global<N, 1, 1, NT, true, SH>(buf, twz, [&](int row, int) {
    return make_float2(xa[row], hasb ? xb[row] : 0.f);
  });
  if (mode == 2) {
#pragma unroll
    for (int j = 0; j < HU; ++j) {
      const int kk = (int)threadIdx.x + j * NT;
      if (kk <= U) {
        const float2 h = PRE ? hv[PRE ? j : 0] : ha[kk];
        const int nk = (N - kk) & (N - 1);
        const int sk = fft::lds_slot<SH>(kk), snk = fft::lds_slot<SH>(nk);
        buf[sk] = cmul(buf[sk], h);
        if (nk != kk) buf[snk] = cmul(buf[snk], conjf2(h));
      }
    }
  } else {
    for (int kk = (int)threadIdx.x; kk <= U; kk += NT) {
      const float2 a = ha[kk], b = hasb ? hb[kk] : make_float2(0.f, 0.f);
      const float2 s = make_float2(0.5f * (a.x + b.x), 0.5f * (a.y + b.y));
      const float2 d = make_float2(0.5f * (a.x - b.x), 0.5f * (a.y - b.y));
      const int nk = (N - kk) & (N - 1);
      const int sk = fft::lds_slot<SH>(kk), snk = fft::lds_slot<SH>(nk);
      const float2 zk = buf[sk], znk = buf[snk];
      buf[sk] = cadd(cmul(zk, s), cmul(conjf2(znk), d));
      if (nk != kk) buf[snk] = cadd(cmul(znk, conjf2(s)), cmul(conjf2(zk), conjf2(d)));
    }
  }
  __syncthreads();
  // outputs U + j -> row j of the pair's columns, in place over the inputs
  // (every input of this workgroup was read in the first pass)
  fft::inverse_to_global<N, 1, 1, NT, true, SH>(buf, twz, [&](int row, int, float2 v) {
    const int j = row - U;
    xa[j] = v.x;
    if (hasb) xb[j] = v.y;
  });
}

// The column tile of 2U = 2 NS points, above the largest transform a column
// can hold in LDS, as two NS-point transforms (U = NS): the even and the odd
// bins of the 2U-point spectrum.  With z[n] the complex column (zero for
// n >= U, so every input row is one of the NS points),
//   Z[2k + p] = DFT_NS(z[n] w_2U^{p n})[k],
// and the outputs U + j of the inverse 2U-point transform of the product are
//   A[j] + w_2U^{-(U + j)} B[j] = A[j] - w_2U^{-j} B[j],
// A and B the NS-point inverses of the even and the odd products.  PAR = 1
// stores -w_2U^{-j} B[j] into Y; PAR = 0, launched after it, stores
// A[j] + Y[j] into X over its own inputs (all read in its first pass).  The
// bins k > U of the filter spectra follow from H[2U - k] = conj(H[k]); for
// pairs of two channels the mirror bin 2U - k of bin k lies in the same half.
template <int NS, int PAR>
__global__ __launch_bounds__(ColCfg<NS>::NT, ColCfg<NS>::MINB) void k_fft_coltile2(
    float* __restrict__ X, float* __restrict__ Y, int ldx, const float2* __restrict__ Hc,
    const float2* __restrict__ tw, long long g0, int ncols, int BD, int D, int B, int mode) {
  constexpr int NT = ColCfg<NS>::NT, U = NS, N = 2 * NS;
  constexpr int SH = ColCfg<NS>::SH;
  static_assert(!ColCfg<NS>::TWL, "two-level twiddles");
  __shared__ float2 buf[ColCfg<NS>::SLOTS];
  __shared__ float2 twl[NS / 64 + 64];
  for (int j = (int)threadIdx.x; j < NS / 64; j += NT) twl[j] = tw[NS + 64 * j];
  for (int l = (int)threadIdx.x; l < 64; l += NT) twl[NS / 64 + l] = tw[NS + l];
  const TwSplit<NS> twz{twl, twl + NS / 64};
  // w_2U^m for m < U, as w_2U^(m mod C) w_32^(m div C) with C = NS/16: the
  // rows of one butterfly share the first factor (one table read each)
  constexpr int C = NS / 16;
  auto w2u = [&](int m) { return cmul(tw[N + (m & (C - 1))], tw[32 + m / C]); };
  int ca, cb;
  col_pair(fft::xcd_logical((int)blockIdx.x, (int)gridDim.x), mode, BD, D, B, ca, cb);
  const bool hasb = cb < ncols;
  float* xa = X + (size_t)ca * ldx;
  float* xb = X + (size_t)(hasb ? cb : ca) * ldx;
  float* ya = Y + (size_t)ca * ldx;
  float* yb = Y + (size_t)(hasb ? cb : ca) * ldx;
  const long long ga = g0 + ca, gb = g0 + (hasb ? cb : ca);
  const long long ma = ga / BD, mb = gb / BD;
  const int da = (int)(ga - ma * BD) % D, db = (int)(gb - mb * BD) % D;
  const float2* ha = Hc + ((size_t)ma * D + da) * (U + 1);
  const float2* hb = Hc + ((size_t)mb * D + db) * (U + 1);

  fft::forward_from_global<NS, 1, 1, NT, false, SH>(buf, twz, [&](int row, int) -> float2 {
    const float2 v = make_float2(xa[row], hasb ? xb[row] : 0.f);
    if constexpr (PAR == 1) return cmul(v, w2u(row));
    return v;
  });
  if (mode == 2) {
    // one channel: P = Z H at every bin k = 2 kk + PAR
    for (int kk = (int)threadIdx.x; kk < NS; kk += NT) {
      const int k = 2 * kk + PAR;
      const float2 h = k <= U ? ha[k] : conjf2(ha[N - k]);
      const int sk = fft::lds_slot<SH>(kk);
      buf[sk] = cmul(buf[sk], h);
    }
  } else {
    // bin k = 2 kk + PAR <= U with its mirror 2U - k = bin (NS - kk - PAR) mod NS
    constexpr int KH = PAR ? NS / 2 : NS / 2 + 1;
    for (int kk = (int)threadIdx.x; kk < KH; kk += NT) {
      const int k = 2 * kk + PAR;
      const int nk = (NS - kk - PAR) & (NS - 1);
      const float2 a = ha[k], b = hasb ? hb[k] : make_float2(0.f, 0.f);
      const float2 s = make_float2(0.5f * (a.x + b.x), 0.5f * (a.y + b.y));
      const float2 d = make_float2(0.5f * (a.x - b.x), 0.5f * (a.y - b.y));
      const int sk = fft::lds_slot<SH>(kk), snk = fft::lds_slot<SH>(nk);
      const float2 zk = buf[sk], znk = buf[snk];
      buf[sk] = cadd(cmul(zk, s), cmul(conjf2(znk), d));
      if (nk != kk) buf[snk] = cadd(cmul(znk, conjf2(s)), cmul(conjf2(zk), conjf2(d)));
    }
  }
  __syncthreads();
  fft::inverse_to_global<NS, 1, 1, NT, false, SH>(buf, twz, [&](int row, int, float2 v) {
    if constexpr (PAR == 1) {
      const float2 b = cmul(v, conjf2(w2u(row)));
      ya[row] = -b.x;
      if (hasb) yb[row] = -b.y;
    } else {
      xa[row] = v.x + ya[row];
      if (hasb) xb[row] = v.y + yb[row];
    }
  });
}

// ---- Column-major mirror tiles.
//
// The mirror C holds, per layer, one row of L complex samples per column
// pair: C[m][p][t] = (y_a[t], y_b[t]) for the positions t whose inputs are
// known, and the large tiles' accumulators for later positions, where
// the pair p is two real columns (a, b) of the layer:
//   batch pairs (B even):  p = q D + d,  a = 2q D + d,  b = a + D  (one channel);
//   adjacent pairs:        a = 2p,  b = 2p + 1 (absent when b = B D).
// Every T0 positions (T0 the smallest mirrored tile side) the inputs of the
// last T0 positions are copied in (k_cm_yin) and, after that position's
// tile, the mirrored accumulators of the next T0 positions are handed to the
// time-major state (k_cm_merge).  The mirrored tiles (k_cm_tile) read their
// U inputs and write their U outputs as contiguous runs of one pair's row.

// Real columns (a, b) of pair p of a layer; b < 0 when absent.
__device__ __forceinline__ void cm_cols(int p, bool bpair, int D, int BD, int& a, int& b) {
  if (bpair) {
    const int q = p / D, d = p - q * D;
    a = 2 * q * D + d;
    b = a + D;
  } else {
    a = 2 * p;
    b = a + 1 < BD ? a + 1 : -1;
  }
}

// Stored pair of the r-th workgroup of a layer in the mirrored tiles: with
// batch pairs, the B/2 pairs of one channel (stored D apart) run on
// consecutive workgroups, so they read that channel's filter spectrum while
// it is in their XCD's L2; adjacent-column pairs keep their order.
__device__ __forceinline__ int cm_pair_of(int r, bool bpair, int PC, int D) {
  if (!bpair) return r;
  const int h = PC / D;  // batch pairs per channel
  const int d = r / h;
  return (r - d * h) * D + d;
}

constexpr int kCmT = 64;  // transpose tile: 64 pairs x 64 positions

// C[m][p][t] = (S[m][t][a], S[m][t][b]) for t in [row0, row1).  Grid (pair
// blocks, position blocks, M); 256 threads.
__global__ __launch_bounds__(kTThreads) void k_cm_yin(const float* __restrict__ S, size_t lstride,
                                                      float2* __restrict__ C, size_t cstride,
                                                      int L, int PC, int BD, int D, int bpair,
                                                      int row0, int row1) {
  __shared__ float2 tile[kCmT][kCmT + 1];
  const int m = (int)blockIdx.z;
  const int p0 = (int)blockIdx.x * kCmT, r0 = row0 + (int)blockIdx.y * kCmT;
  const int x = (int)threadIdx.x & (kCmT - 1), y4 = (int)threadIdx.x / kCmT;
  const float* Sm = S + (size_t)m * lstride;
  {
    const int p = p0 + x;
    int a = 0, b = -1;
    if (p < PC) cm_cols(p, bpair != 0, D, BD, a, b);
#pragma unroll
    for (int k = 0; k < kCmT / 4; ++k) {
      const int r = y4 + 4 * k, t = r0 + r;
      if (p < PC && t < row1) {
        const float* row = Sm + (size_t)t * BD;
        tile[r][x] = make_float2(row[a], b >= 0 ? row[b] : 0.f);
      }
    }
  }
  __syncthreads();
  float2* Cm = C + (size_t)m * cstride;
#pragma unroll
  for (int k = 0; k < kCmT / 4; ++k) {
    const int xx = y4 + 4 * k, p = p0 + xx, t = r0 + x;
    if (p < PC && t < row1) Cm[(size_t)p * L + t] = tile[x][xx];
  }
}

// S[m][t][a] (+)= C[m][p][t].x and S[m][t][b] (+)= C[m][p][t].y for t in
// [row0, row1): stored when STORE (the rows hold nothing else yet), added
// otherwise.
template <bool STORE>
__global__ __launch_bounds__(kTThreads) void k_cm_merge(const float2* __restrict__ C,
                                                        size_t cstride, float* __restrict__ S,
                                                        size_t lstride, int L, int PC, int BD,
                                                        int D, int bpair, int row0, int row1) {
  __shared__ float2 tile[kCmT][kCmT + 1];
  const int m = (int)blockIdx.z;
  const int p0 = (int)blockIdx.x * kCmT, r0 = row0 + (int)blockIdx.y * kCmT;
  const int x = (int)threadIdx.x & (kCmT - 1), y4 = (int)threadIdx.x / kCmT;
  const float2* Cm = C + (size_t)m * cstride;
#pragma unroll
  for (int k = 0; k < kCmT / 4; ++k) {
    const int xx = y4 + 4 * k, p = p0 + xx, t = r0 + x;
    if (p < PC && t < row1) tile[x][xx] = Cm[(size_t)p * L + t];
  }
  __syncthreads();
  const int p = p0 + x;
  if (p >= PC) return;
  int a, b;
  cm_cols(p, bpair != 0, D, BD, a, b);
  float* Sm = S + (size_t)m * lstride;
#pragma unroll
  for (int k = 0; k < kCmT / 4; ++k) {
    const int r = y4 + 4 * k, t = r0 + r;
    if (t < row1) {
      float* row = Sm + (size_t)t * BD;
      const float2 v = tile[r][x];
      row[a] = STORE ? v.x : row[a] + v.x;
      if (b >= 0) row[b] = STORE ? v.y : row[b] + v.y;
    }
  }
}

// The two mirror copies with 16-byte accesses, for shapes where a block of 64
// pairs has its first columns in one 256-byte run of a state row and its
// second columns in another (batch pairs with D a multiple of 64) or all of
// them in one 512-byte run (neighbouring columns with B*D a multiple of 128):
// a lane moves four pairs of a row, or two positions of a pair, at once.
__device__ __forceinline__ void cm_block_cols(int p0, bool bpair, int D, int& a0, int& b0) {
  if (bpair) {
    const int q = p0 / D, d0 = p0 - q * D;
    a0 = 2 * q * D + d0;
    b0 = a0 + D;
  } else {
    a0 = 2 * p0;
    b0 = -1;
  }
}

// Pairs 4g .. 4g+3 of the block at row `row`: (a, b) of each.
__device__ __forceinline__ void cm_load4(const float* __restrict__ row, int a0, int b0, int g,
                                         float2 (&v)[4]) {
  if (b0 >= 0) {
    const float4 A = *reinterpret_cast<const float4*>(row + a0 + 4 * g);
    const float4 B = *reinterpret_cast<const float4*>(row + b0 + 4 * g);
    v[0] = make_float2(A.x, B.x);
    v[1] = make_float2(A.y, B.y);
    v[2] = make_float2(A.z, B.z);
    v[3] = make_float2(A.w, B.w);
  } else {
    const float4 P = *reinterpret_cast<const float4*>(row + a0 + 8 * g);
    const float4 Q = *reinterpret_cast<const float4*>(row + a0 + 8 * g + 4);
    v[0] = make_float2(P.x, P.y);
    v[1] = make_float2(P.z, P.w);
    v[2] = make_float2(Q.x, Q.y);
    v[3] = make_float2(Q.z, Q.w);
  }
}

template <bool STORE>
__device__ __forceinline__ void cm_store4(float* row, int a0, int b0, int g, const float2 (&v)[4]) {
  if (b0 >= 0) {
    float4* pa = reinterpret_cast<float4*>(row + a0 + 4 * g);
    float4* pb = reinterpret_cast<float4*>(row + b0 + 4 * g);
    float4 A = make_float4(v[0].x, v[1].x, v[2].x, v[3].x);
    float4 B = make_float4(v[0].y, v[1].y, v[2].y, v[3].y);
    if constexpr (!STORE) {
      const float4 oa = *pa, ob = *pb;
      A = make_float4(oa.x + A.x, oa.y + A.y, oa.z + A.z, oa.w + A.w);
      B = make_float4(ob.x + B.x, ob.y + B.y, ob.z + B.z, ob.w + B.w);
    }
    *pa = A;
    *pb = B;
  } else {
    float4* pp = reinterpret_cast<float4*>(row + a0 + 8 * g);
    float4 P = make_float4(v[0].x, v[0].y, v[1].x, v[1].y);
    float4 Q = make_float4(v[2].x, v[2].y, v[3].x, v[3].y);
    if constexpr (!STORE) {
      const float4 op = pp[0], oq = pp[1];
      P = make_float4(op.x + P.x, op.y + P.y, op.z + P.z, op.w + P.w);
      Q = make_float4(oq.x + Q.x, oq.y + Q.y, oq.z + Q.z, oq.w + Q.w);
    }
    pp[0] = P;
    pp[1] = Q;
  }
}

// k_cm_yin with 16-byte accesses.  Phase 1: lane (g = lane & 15, r) reads
// four pairs of rows r, r+16, r+32, r+48; phase 2: each group of 32 lanes
// writes the 64 positions of one pair as 32 float4 (two positions each).
__global__ __launch_bounds__(kTThreads) void k_cm_yin4(const float* __restrict__ S, size_t lstride,
                                                       float2* __restrict__ C, size_t cstride,
                                                       int L, int BD, int D, int bpair, int row0,
                                                       int row1) {
  __shared__ float2 tile[kCmT][kCmT + 1];
  const int m = (int)blockIdx.z;
  const int p0 = (int)blockIdx.x * kCmT, r0 = row0 + (int)blockIdx.y * kCmT;
  int a0, b0;
  cm_block_cols(p0, bpair != 0, D, a0, b0);
  const float* Sm = S + (size_t)m * lstride;
  {
    const int g = (int)threadIdx.x & 15, r16 = (int)threadIdx.x >> 4;
#pragma unroll
    for (int k = 0; k < kCmT / 16; ++k) {
      const int r = r16 + 16 * k;
      if (r0 + r < row1) {
        float2 v[4];
        cm_load4(Sm + (size_t)(r0 + r) * BD, a0, b0, g, v);
#pragma unroll
        for (int j = 0; j < 4; ++j) tile[r][4 * g + j] = v[j];
      }
    }
  }
  __syncthreads();
  float2* Cm = C + (size_t)m * cstride;
  const int l = (int)threadIdx.x & 31, grp = (int)threadIdx.x >> 5;
#pragma unroll
  for (int k = 0; k < kCmT / 8; ++k) {
    const int x = grp + 8 * k, t = r0 + 2 * l;
    if (t + 1 < row1) {
      const float2 u = tile[2 * l][x], w = tile[2 * l + 1][x];
      *reinterpret_cast<float4*>(Cm + (size_t)(p0 + x) * L + t) = make_float4(u.x, u.y, w.x, w.y);
    } else if (t < row1) {
      Cm[(size_t)(p0 + x) * L + t] = tile[2 * l][x];
    }
  }
}

// k_cm_merge with 16-byte accesses (the reverse of k_cm_yin4).
template <bool STORE>
__global__ __launch_bounds__(kTThreads) void k_cm_merge4(const float2* __restrict__ C,
                                                         size_t cstride, float* __restrict__ S,
                                                         size_t lstride, int L, int BD, int D,
                                                         int bpair, int row0, int row1) {
  __shared__ float2 tile[kCmT][kCmT + 1];
  const int m = (int)blockIdx.z;
  const int p0 = (int)blockIdx.x * kCmT, r0 = row0 + (int)blockIdx.y * kCmT;
  const float2* Cm = C + (size_t)m * cstride;
  {
    const int l = (int)threadIdx.x & 31, grp = (int)threadIdx.x >> 5;
#pragma unroll
    for (int k = 0; k < kCmT / 8; ++k) {
      const int x = grp + 8 * k, t = r0 + 2 * l;
      if (t + 1 < row1) {
        const float4 v = *reinterpret_cast<const float4*>(Cm + (size_t)(p0 + x) * L + t);
        tile[2 * l][x] = make_float2(v.x, v.y);
        tile[2 * l + 1][x] = make_float2(v.z, v.w);
      } else if (t < row1) {
        tile[2 * l][x] = Cm[(size_t)(p0 + x) * L + t];
      }
    }
  }
  __syncthreads();
  int a0, b0;
  cm_block_cols(p0, bpair != 0, D, a0, b0);
  float* Sm = S + (size_t)m * lstride;
  const int g = (int)threadIdx.x & 15, r16 = (int)threadIdx.x >> 4;
#pragma unroll
  for (int k = 0; k < kCmT / 16; ++k) {
    const int r = r16 + 16 * k;
    if (r0 + r < row1) {
      float2 v[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) v[j] = tile[r][4 * g + j];
      cm_store4<STORE>(Sm + (size_t)(r0 + r) * BD, a0, b0, g, v);
    }
  }
}

// Spectral product of the transform in buf (padded LDS, one column) for a
// pair: one channel (spectrum ha, plain P = Z H over bins k <= U and their
// mirrors) or two (ha, hb: P[k] = Z[k] S[k] + conj(Z[N-k]) D[k]).  hv: ha
// preloaded into registers (PRE).  Synchronises at the end.
template <int N, bool PRE, int HU>
__device__ __forceinline__ void cm_product(float2* buf, bool one, const float2* __restrict__ ha,
                                           const float2* __restrict__ hb, bool hasb,
                                           const float2 (&hv)[PRE ? HU : 1]) {
  constexpr int NT = ColCfg<N>::NT, U = N / 2, SH = ColCfg<N>::SH;
  if (one) {
#pragma unroll
    for (int j = 0; j < HU; ++j) {
      const int kk = (int)threadIdx.x + j * NT;
      if (kk <= U) {
        const float2 h = PRE ? hv[PRE ? j : 0] : ha[kk];
        const int nk = (N - kk) & (N - 1);
        const int sk = fft::lds_slot<SH>(kk), snk = fft::lds_slot<SH>(nk);
        buf[sk] = cmul(buf[sk], h);
        if (nk != kk) buf[snk] = cmul(buf[snk], conjf2(h));
      }
    }
  } else {
    for (int kk = (int)threadIdx.x; kk <= U; kk += NT) {
      const float2 a = ha[kk], b = hasb ? hb[kk] : make_float2(0.f, 0.f);
      const float2 s = make_float2(0.5f * (a.x + b.x), 0.5f * (a.y + b.y));
      const float2 d = make_float2(0.5f * (a.x - b.x), 0.5f * (a.y - b.y));
      const int nk = (N - kk) & (N - 1);
      const int sk = fft::lds_slot<SH>(kk), snk = fft::lds_slot<SH>(nk);
      const float2 zk = buf[sk], znk = buf[snk];
      buf[sk] = cadd(cmul(zk, s), cmul(conjf2(znk), d));
      if (nk != kk) buf[snk] = cadd(cmul(znk, conjf2(s)), cmul(conjf2(zk), conjf2(d)));
    }
  }
  __syncthreads();
}

// Mirrored tile of side U = N/2 at position i for every pair of every layer
// (one workgroup per pair, the same transform as k_fft_coltile): inputs
// C[p][i-U .. i), outputs j < dst_len into C[p][i+j], stored when `store`
// (no earlier mirrored tile reached those positions) and added otherwise.
template <int N>
__global__ __launch_bounds__(ColCfg<N>::NT, ColCfg<N>::MINB) void k_cm_tile(
    float2* __restrict__ C, size_t cstride, int L, const float2* __restrict__ Hc,
    const float2* __restrict__ tw, int PC, int BD, int D, int bpair, int i, int dst_len,
    int store) {
  constexpr int NT = ColCfg<N>::NT, U = N / 2;
  constexpr int HU = (U + 1 + NT - 1) / NT;
  constexpr bool PRE = N <= 8192;
  using TW = typename std::conditional<ColCfg<N>::TWL, fft::TwLds<N>, TwSplit<N>>::type;
  constexpr int SH = ColCfg<N>::SH;
  __shared__ float2 buf[ColCfg<N>::SLOTS];
  __shared__ float2 twl[ColCfg<N>::TWL ? N : N / 64 + 64];
  TW twz;
  if constexpr (ColCfg<N>::TWL) {
    fft::load_twiddles<N, NT>(twl, tw);
    twz = TW{twl};
  } else {
    for (int j = (int)threadIdx.x; j < N / 64; j += NT) twl[j] = tw[N + 64 * j];
    for (int l = (int)threadIdx.x; l < 64; l += NT) twl[N / 64 + l] = tw[N + l];
    twz = TW{twl, twl + N / 64};
  }
  const int g = fft::xcd_logical((int)blockIdx.x, (int)gridDim.x);
  const int m = g / PC, p = cm_pair_of(g - m * PC, bpair != 0, PC, D);
  int a, b;
  cm_cols(p, bpair != 0, D, BD, a, b);
  const bool one = bpair != 0;
  const float2* ha = Hc + ((size_t)m * D + a % D) * (U + 1);
  const float2* hb = Hc + ((size_t)m * D + (b >= 0 ? b : a) % D) * (U + 1);
  float2 hv[PRE ? HU : 1];
  if constexpr (PRE) {
    if (one) {
#pragma unroll
      for (int j = 0; j < HU; ++j) {
        const int kk = (int)threadIdx.x + j * NT;
        hv[j] = kk <= U ? ha[kk] : make_float2(0.f, 0.f);
      }
    }
  }
  float2* col = C + (size_t)m * cstride + (size_t)p * L;
  const float2* in = col + (i - U);
  fft::forward_from_global<N, 1, 1, NT, true, SH>(buf, twz, [&](int row, int) { return in[row]; });
  cm_product<N, PRE, HU>(buf, one, ha, hb, b >= 0, hv);
  float2* out = col + i;
  fft::inverse_to_global<N, 1, 1, NT, true, SH>(buf, twz, [&](int row, int, float2 v) {
    const int j = row - U;
    if (j < dst_len) out[j] = store ? v : cadd(out[j], v);
  });
}

// The mirrored tile of 2U = 2 NS (above one column's LDS transform) as two
// NS-point halves, the even and the odd bins (see k_fft_coltile2), for the
// pairs [g0, g0 + npairs) of all layers: PAR = 1 stores -w_2U^{-j} B[j] into
// Y[pair - g0][j]; PAR = 0, launched after it, adds A[j] + Y into the
// outputs.
template <int NS, int PAR>
__global__ __launch_bounds__(ColCfg<NS>::NT, ColCfg<NS>::MINB) void k_cm_tile2(
    float2* __restrict__ C, size_t cstride, int L, float2* __restrict__ Y,
    const float2* __restrict__ Hc, const float2* __restrict__ tw, int PC, int BD, int D,
    int bpair, int i, int dst_len, int store, int g0) {
  constexpr int NT = ColCfg<NS>::NT, U = NS, N = 2 * NS;
  constexpr int SH = ColCfg<NS>::SH;
  static_assert(!ColCfg<NS>::TWL, "two-level twiddles");
  __shared__ float2 buf[ColCfg<NS>::SLOTS];
  __shared__ float2 twl[NS / 64 + 64];
  for (int j = (int)threadIdx.x; j < NS / 64; j += NT) twl[j] = tw[NS + 64 * j];
  for (int l = (int)threadIdx.x; l < 64; l += NT) twl[NS / 64 + l] = tw[NS + l];
  const TwSplit<NS> twz{twl, twl + NS / 64};
  constexpr int CC = NS / 16;
  auto w2u = [&](int mm) { return cmul(tw[N + (mm & (CC - 1))], tw[32 + mm / CC]); };
  const int gl = fft::xcd_logical((int)blockIdx.x, (int)gridDim.x);
  const int g = g0 + gl;
  const int m = g / PC, p = cm_pair_of(g - m * PC, bpair != 0, PC, D);
  int a, b;
  cm_cols(p, bpair != 0, D, BD, a, b);
  const bool hasb = b >= 0;
  const float2* ha = Hc + ((size_t)m * D + a % D) * (U + 1);
  const float2* hb = Hc + ((size_t)m * D + (hasb ? b : a) % D) * (U + 1);
  float2* col = C + (size_t)m * cstride + (size_t)p * L;
  const float2* in = col + (i - U);
  float2* y = Y + (size_t)gl * U;
  fft::forward_from_global<NS, 1, 1, NT, false, SH>(buf, twz, [&](int row, int) -> float2 {
    const float2 v = in[row];
    if constexpr (PAR == 1) return cmul(v, w2u(row));
    return v;
  });
  if (bpair) {
    for (int kk = (int)threadIdx.x; kk < NS; kk += NT) {
      const int k = 2 * kk + PAR;
      const float2 h = k <= U ? ha[k] : conjf2(ha[N - k]);
      const int sk = fft::lds_slot<SH>(kk);
      buf[sk] = cmul(buf[sk], h);
    }
  } else {
    constexpr int KH = PAR ? NS / 2 : NS / 2 + 1;
    for (int kk = (int)threadIdx.x; kk < KH; kk += NT) {
      const int k = 2 * kk + PAR;
      const int nk = (NS - kk - PAR) & (NS - 1);
      const float2 av = ha[k], bv = hasb ? hb[k] : make_float2(0.f, 0.f);
      const float2 s = make_float2(0.5f * (av.x + bv.x), 0.5f * (av.y + bv.y));
      const float2 d = make_float2(0.5f * (av.x - bv.x), 0.5f * (av.y - bv.y));
      const int sk = fft::lds_slot<SH>(kk), snk = fft::lds_slot<SH>(nk);
      const float2 zk = buf[sk], znk = buf[snk];
      buf[sk] = cadd(cmul(zk, s), cmul(conjf2(znk), d));
      if (nk != kk) buf[snk] = cadd(cmul(znk, conjf2(s)), cmul(conjf2(zk), conjf2(d)));
    }
  }
  __syncthreads();
  float2* out = col + i;
  fft::inverse_to_global<NS, 1, 1, NT, false, SH>(buf, twz, [&](int row, int, float2 v) {
    if constexpr (PAR == 1) {
      const float2 bb = cmul(v, conjf2(w2u(row)));
      y[row] = make_float2(-bb.x, -bb.y);
    } else {
      if (row < dst_len) {
        const float2 o = cadd(v, y[row]);
        out[row] = store ? o : cadd(out[row], o);
      }
    }
  });
}

}  // namespace

int fft_col_chunk(int U, size_t scratch_bytes, long long total_cols) {
  long long cap = (long long)(scratch_bytes / (sizeof(float) * (size_t)U));
  cap = cap / kTT * kTT;
  const long long need = (total_cols + kTT - 1) / kTT * kTT;
  if (cap > need) cap = need;
  if (cap > (1LL << 30)) cap = 1LL << 30;
  return (int)cap;
}

hipError_t launch_fft_col_tile(float* S, const float2* Hc, const float2* tw, const Shape& s, int i,
                               int U, int dst_len, float2* scratch, size_t scratch_bytes,
                               hipStream_t st, bool in_place) {
  if (dst_len <= 0) return hipSuccess;
  const int N = 2 * U;
  const long long total = (long long)s.M * s.BD;
  // above one column's LDS transform: two halves (k_fft_coltile2), with a
  // second U floats per column in the scratch for the odd half's outputs
  const bool split = N > kMaxColFftN1;
  int chunk = fft_col_chunk(U, split ? scratch_bytes / 2 : scratch_bytes, total);
  if (chunk <= 0) return hipErrorOutOfMemory;
  // whole layers per chunk where possible (then the pairs and their order can
  // follow the spectra: see k_fft_coltile)
  const bool layers = s.BD % 64 == 0 && chunk >= s.BD;
  if (layers) chunk = chunk / s.BD * s.BD;
  const int mode = layers && s.B % 2 == 0 ? 2 : (layers && s.D % 2 == 0 ? 1 : 0);
  float* X = reinterpret_cast<float*>(scratch);
  float* Y = X + (size_t)chunk * U;  // the odd half's outputs (split tiles only)
  const size_t lstride = (size_t)s.SL * s.BD;
  // 16-byte transposes: whole float4s in one layer's rows (B*D, and with it
  // every chunk start, a multiple of 4) and in the columns (U and the rows
  // moved back multiples of 4)
  const bool vin = s.BD % 4 == 0 && U % 4 == 0;
  const bool vout = vin && dst_len % 4 == 0;
  for (long long g0 = 0; g0 < total; g0 += chunk) {
    const int nc = (int)(total - g0 < chunk ? total - g0 : chunk);
    const dim3 tin((unsigned)((nc + kTT - 1) / kTT), (unsigned)((U + kTT - 1) / kTT));
    if (vin)
      hipLaunchKernelGGL(k_rows_to_cols4, tin, dim3(kTThreads), 0, st, S, lstride, s.BD, i - U, U,
                         g0, nc, X, U);
    else
      hipLaunchKernelGGL(k_rows_to_cols, tin, dim3(kTThreads), 0, st, S, lstride, s.BD, i - U, U,
                         g0, nc, X, U);
    const dim3 grid((unsigned)((nc + 1) / 2));
    switch (N) {
#define LCSM_CASE(NN)                                                                            \
  case NN:                                                                                       \
    hipLaunchKernelGGL(k_fft_coltile<NN>, grid, dim3(ColCfg<NN>::NT), 0, st, X, U, Hc, tw, g0, nc, \
                       s.BD, s.D, s.B, mode);                                                    \
    break;
      LCSM_CASE(4) LCSM_CASE(8) LCSM_CASE(16) LCSM_CASE(32) LCSM_CASE(64) LCSM_CASE(128)
      LCSM_CASE(256) LCSM_CASE(512) LCSM_CASE(1024) LCSM_CASE(2048) LCSM_CASE(4096)
      LCSM_CASE(8192) LCSM_CASE(16384)
#undef LCSM_CASE
      case 2 * kMaxColFftN1:
        hipLaunchKernelGGL((k_fft_coltile2<kMaxColFftN1, 1>), grid, dim3(ColCfg<kMaxColFftN1>::NT), 0,
                           st, X, Y, U, Hc, tw, g0, nc, s.BD, s.D, s.B, mode);
        hipLaunchKernelGGL((k_fft_coltile2<kMaxColFftN1, 0>), grid, dim3(ColCfg<kMaxColFftN1>::NT), 0,
                           st, X, Y, U, Hc, tw, g0, nc, s.BD, s.D, s.B, mode);
        break;
      default:
        return hipErrorInvalidValue;
    }
    const dim3 tout((unsigned)((nc + kTT - 1) / kTT), (unsigned)((dst_len + kTT - 1) / kTT));
    if (in_place && vout)
      hipLaunchKernelGGL(k_cols_to_rows4<true>, tout, dim3(kTThreads), 0, st, X, U, S, lstride,
                         s.BD, i - U, dst_len, g0, nc);
    else if (in_place)
      hipLaunchKernelGGL(k_cols_to_rows<true>, tout, dim3(kTThreads), 0, st, X, U, S, lstride, s.BD,
                         i - U, dst_len, g0, nc);
    else if (vout)
      hipLaunchKernelGGL(k_cols_to_rows4<false>, tout, dim3(kTThreads), 0, st, X, U, S, lstride,
                         s.BD, i, dst_len, g0, nc);
    else
      hipLaunchKernelGGL(k_cols_to_rows<false>, tout, dim3(kTThreads), 0, st, X, U, S, lstride, s.BD,
                         i, dst_len, g0, nc);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// 16-byte mirror copies: every block of 64 pairs lies in whole aligned runs
// (and L even keeps the two positions of a float4 in one pair's row).
static bool cm_vec(const Shape& s, const CmShape& cm) {
  if (s.L % 2 != 0) return false;
  return cm.bpair ? s.D % kCmT == 0 : s.BD % (2 * kCmT) == 0;
}

hipError_t launch_cm_yin(const float* S, float2* C, const Shape& s, const CmShape& cm, int row0,
                         int row1, hipStream_t st) {
  if (row1 <= row0) return hipSuccess;
  const dim3 grid((unsigned)((cm.PC + kCmT - 1) / kCmT), (unsigned)((row1 - row0 + kCmT - 1) / kCmT),
                  (unsigned)s.M);
  if (cm_vec(s, cm) && row0 % 2 == 0)
    hipLaunchKernelGGL(k_cm_yin4, grid, dim3(kTThreads), 0, st, S, (size_t)s.SL * s.BD, C,
                       (size_t)cm.PC * s.L, s.L, s.BD, s.D, cm.bpair, row0, row1);
  else
    hipLaunchKernelGGL(k_cm_yin, grid, dim3(kTThreads), 0, st, S, (size_t)s.SL * s.BD, C,
                       (size_t)cm.PC * s.L, s.L, cm.PC, s.BD, s.D, cm.bpair, row0, row1);
  return hipGetLastError();
}

hipError_t launch_cm_merge(const float2* C, float* S, const Shape& s, const CmShape& cm, int row0,
                           int row1, bool store, hipStream_t st) {
  if (row1 <= row0) return hipSuccess;
  const dim3 grid((unsigned)((cm.PC + kCmT - 1) / kCmT), (unsigned)((row1 - row0 + kCmT - 1) / kCmT),
                  (unsigned)s.M);
  const bool vec = cm_vec(s, cm) && row0 % 2 == 0;
  if (vec && store)
    hipLaunchKernelGGL(k_cm_merge4<true>, grid, dim3(kTThreads), 0, st, C, (size_t)cm.PC * s.L, S,
                       (size_t)s.SL * s.BD, s.L, s.BD, s.D, cm.bpair, row0, row1);
  else if (vec)
    hipLaunchKernelGGL(k_cm_merge4<false>, grid, dim3(kTThreads), 0, st, C, (size_t)cm.PC * s.L, S,
                       (size_t)s.SL * s.BD, s.L, s.BD, s.D, cm.bpair, row0, row1);
  else if (store)
    hipLaunchKernelGGL(k_cm_merge<true>, grid, dim3(kTThreads), 0, st, C, (size_t)cm.PC * s.L, S,
                       (size_t)s.SL * s.BD, s.L, cm.PC, s.BD, s.D, cm.bpair, row0, row1);
  else
    hipLaunchKernelGGL(k_cm_merge<false>, grid, dim3(kTThreads), 0, st, C, (size_t)cm.PC * s.L, S,
                       (size_t)s.SL * s.BD, s.L, cm.PC, s.BD, s.D, cm.bpair, row0, row1);
  return hipGetLastError();
}

hipError_t launch_cm_tile(float2* C, const float2* Hc, const float2* tw, const Shape& s,
                          const CmShape& cm, int i, int U, int dst_len, bool store, float2* scratch,
                          size_t scratch_bytes, hipStream_t st) {
  if (dst_len <= 0) return hipSuccess;
  const int N = 2 * U;
  const long long total = (long long)s.M * cm.PC;
  const size_t cstride = (size_t)cm.PC * s.L;
  if (N <= kMaxColFftN1) {
    const dim3 grid((unsigned)total);
    switch (N) {
#define LCSM_CM_CASE(NN)                                                                      \
  case NN:                                                                                    \
    hipLaunchKernelGGL(k_cm_tile<NN>, grid, dim3(ColCfg<NN>::NT), 0, st, C, cstride, s.L, Hc, \
                       tw, cm.PC, s.BD, s.D, cm.bpair, i, dst_len, store ? 1 : 0);            \
    break;
      LCSM_CM_CASE(4) LCSM_CM_CASE(8) LCSM_CM_CASE(16) LCSM_CM_CASE(32) LCSM_CM_CASE(64)
      LCSM_CM_CASE(128) LCSM_CM_CASE(256) LCSM_CM_CASE(512) LCSM_CM_CASE(1024)
      LCSM_CM_CASE(2048) LCSM_CM_CASE(4096) LCSM_CM_CASE(8192) LCSM_CM_CASE(16384)
#undef LCSM_CM_CASE
      default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  if (N != 2 * kMaxColFftN1) return hipErrorInvalidValue;
  // the odd half's outputs, U complex values per pair, in the scratch
  const long long chunk = (long long)(scratch_bytes / (sizeof(float2) * (size_t)U));
  if (chunk <= 0) return hipErrorOutOfMemory;
  for (long long g0 = 0; g0 < total; g0 += chunk) {
    const int np = (int)(total - g0 < chunk ? total - g0 : chunk);
    const dim3 grid((unsigned)np);
    hipLaunchKernelGGL((k_cm_tile2<kMaxColFftN1, 1>), grid, dim3(ColCfg<kMaxColFftN1>::NT), 0, st,
                       C, cstride, s.L, scratch, Hc, tw, cm.PC, s.BD, s.D, cm.bpair, i, dst_len,
                       store ? 1 : 0, (int)g0);
    hipLaunchKernelGGL((k_cm_tile2<kMaxColFftN1, 0>), grid, dim3(ColCfg<kMaxColFftN1>::NT), 0, st,
                       C, cstride, s.L, scratch, Hc, tw, cm.PC, s.BD, s.D, cm.bpair, i, dst_len,
                       store ? 1 : 0, (int)g0);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace lcsm
