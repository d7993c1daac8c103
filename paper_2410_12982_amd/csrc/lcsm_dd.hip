// Relaxed online convolution with data-dependent filters (the appendix on
// data-dependent filters, Alg. 5), for gfx950.
//
// State: Y[m][t][c] and R[m][t][c] (c = b*D + d, time-major like the
// data-independent state).  Rows < t of Y hold the inputs y, rows >= t the
// accumulators of the outputs not yet emitted (they share the rows, as in
// the data-independent state); rows < t of R hold rho (rows >= t unused
// until written).
//
// Step t: the red cell z_t = acc_t + y_t rho_0 + y_0 rho_t (last term for
// t >= 1), then for every power of two U dividing t+1 with 2U <= t+1 one
// parallelogram tile of all layers:
//   square (t+1 = 2U):  acc[2U + j] += sum_k yF[k] rF[j-k]
//   rectangle:          acc[t+1 + j] += sum_k yF[k] rR[j-k] + rF[k] yR[j-k]
// for j < 2U-1 (clipped at L), with F the fixed block [U, 2U) and R the
// recent block [t-U+1, t+1) (k and j-k in [0, U)).
#include <stdio.h>
#include <string.h>

#include <new>

#include "lcsm_dd.h"
#include "lcsm_fft_core.h"
#include "lcsm_internal.h"

namespace lcsm {
namespace {

using fft::cadd;
using fft::cmul;
using fft::conjf2;
using fft::csub;

constexpr int kThreads = 256;
constexpr int kDdJ = 16;            // outputs per thread of the direct tile
constexpr int kDdDefaultDirectMaxU = 32;
constexpr int kDdFusedMaxU = 8;      // tiles fused with the red cell

// Contributions of the tile of side U of step t (t + 1 a multiple of U,
// 2U <= t + 1) to the destination rows t + 1 + j, j < 2U - 1, added into dz
// in that order.  fy, fr: the rows 1 .. 2 UMAX - 1 of y and rho (index =
// row); wy, wr: the rows t - UMAX + 1 .. t (index i = row - t + UMAX - 1).
// The square tile (t + 1 = 2U) has the fixed block as its recent block and
// one product.
template <int U, int UMAX>
__device__ __forceinline__ void dd_tile_regs(const float* fy, const float* fr, const float* wy,
                                             const float* wr, float* dz, bool square) {
#pragma unroll
  for (int j = 0; j < 2 * U - 1; ++j) {
    float sum = 0.f;
    if (square) {
#pragma unroll
      for (int k = 0; k < U; ++k)
        if (j - k >= 0 && j - k < U) sum = fmaf(fy[U + k], fr[U + j - k], sum);
    } else {
#pragma unroll
      for (int k = 0; k < U; ++k) {
        if (j - k >= 0 && j - k < U) {
          // recent row t - U + 1 + (j - k) is window index UMAX - U + (j - k)
          sum = fmaf(fy[U + k], wr[UMAX - U + j - k], sum);
          sum = fmaf(fr[U + k], wy[UMAX - U + j - k], sum);
        }
      }
    }
    dz[j] += sum;
  }
}

// Red cell at position t fused with the tiles of every U <= UMAX of step t
// (U | t+1, 2U <= t+1), one thread per column.  Every value the step reads
// -- y_0, rho_0 and the accumulator of row t, the fixed rows 1 .. 2UMAX-1,
// the recent rows t-UMAX+1 .. t-1 (row t is the new input, in registers) and
// the destination rows t+1 .. t+2UMAX-1 -- is loaded before the first store
// (one memory round trip; destination rows past L clamped and not stored).
// The tiles' sums are added into the destination in increasing U, as
// separate read-modify-writes per tile would.
template <int UMAX>
__global__ __launch_bounds__(kThreads) void k_dd_step(const float* __restrict__ y,
                                                      const float* __restrict__ rho,
                                                      float* __restrict__ z, float* __restrict__ Y,
                                                      float* __restrict__ R, int L, int BD, int t) {
  const int c = (int)blockIdx.x * kThreads + (int)threadIdx.x;
  if (c >= BD) return;
  const int m = (int)blockIdx.y;
  const size_t e = (size_t)m * BD + c;
  const size_t rs = (size_t)BD;
  float* ycol = Y + (size_t)m * L * BD + c;
  float* rcol = R + (size_t)m * L * BD + c;
  const float yt = y[e], rt = rho[e];
  const float acc = ycol[(size_t)t * rs];
  const float y0 = ycol[0], r0 = rcol[0];
  constexpr int NF = UMAX > 0 ? 2 * UMAX : 1;
  constexpr int NW = UMAX > 0 ? UMAX : 1;
  constexpr int ND = UMAX > 0 ? 2 * UMAX - 1 : 1;
  float fy[NF], fr[NF], wy[NW], wr[NW], dz[ND];
  if constexpr (UMAX > 0) {
#pragma unroll
    for (int row = 1; row < 2 * UMAX; ++row) {
      const float vy = ycol[(size_t)row * rs], vr = rcol[(size_t)row * rs];
      fy[row] = row == t ? yt : vy;  // row t (the square tile's last fixed row) is the new input
      fr[row] = row == t ? rt : vr;
    }
#pragma unroll
    for (int i = 0; i < UMAX - 1; ++i) {
      const size_t row = (size_t)(t - UMAX + 1 + i);
      wy[i] = ycol[row * rs];
      wr[i] = rcol[row * rs];
    }
    wy[UMAX - 1] = yt;
    wr[UMAX - 1] = rt;
#pragma unroll
    for (int j = 0; j < 2 * UMAX - 1; ++j) {
      const int row = t + 1 + j;
      dz[j] = ycol[(size_t)(row < L ? row : L - 1) * rs];
    }
  }
  z[e] = t == 0 ? fmaf(yt, rt, acc) : fmaf(yt, r0, fmaf(y0, rt, acc));
  ycol[(size_t)t * rs] = yt;
  rcol[(size_t)t * rs] = rt;
  if constexpr (UMAX > 0) {
    // only the largest tile can be the square one (t + 1 = 2 UMAX)
    const bool sq = t + 1 == 2 * UMAX;
    if constexpr (UMAX >= 1) dd_tile_regs<1, UMAX>(fy, fr, wy, wr, dz, sq && UMAX == 1);
    if constexpr (UMAX >= 2) dd_tile_regs<2, UMAX>(fy, fr, wy, wr, dz, sq && UMAX == 2);
    if constexpr (UMAX >= 4) dd_tile_regs<4, UMAX>(fy, fr, wy, wr, dz, sq && UMAX == 4);
    if constexpr (UMAX >= 8) dd_tile_regs<8, UMAX>(fy, fr, wy, wr, dz, sq && UMAX == 8);
#pragma unroll
    for (int j = 0; j < 2 * UMAX - 1; ++j)
      if (t + 1 + j < L) ycol[(size_t)(t + 1 + j) * rs] = dz[j];
  }
}

// Direct parallelogram tile of side U for all layers: thread = (column c,
// outputs j0 .. j0+J-1, layer m).  The recent-block values needed at fixed
// index k form a window j0+jj-k that slides down by one per k, so each k
// loads the two fixed values and the two recent values entering the window.
// SQ: the square tile (recent block = fixed block, one product).
template <int J, bool SQ>
__global__ __launch_bounds__(kThreads) void k_dd_direct(float* __restrict__ Y,
                                                        const float* __restrict__ R, int L,
                                                        int BD, int U, int lo, int d0,
                                                        int dlen) {
  const int c = (int)blockIdx.x * kThreads + (int)threadIdx.x;
  const int j0 = (int)blockIdx.y * J;
  const int m = (int)blockIdx.z;
  if (c >= BD || j0 >= dlen) return;
  const size_t rs = (size_t)BD;
  float* ycol = Y + (size_t)m * L * BD + c;
  const float* rcol = R + (size_t)m * L * BD + c;
  const float* yR = ycol + (size_t)lo * rs;  // recent block (= fixed block for SQ)
  const float* rR = rcol + (size_t)lo * rs;
  const float* yF = ycol + (size_t)U * rs;
  const float* rF = rcol + (size_t)U * rs;

  float acc[J], wy[J], wr[J];  // wy[jj] = yR[j0+jj-k], wr[jj] = rR[j0+jj-k]
#pragma unroll
  for (int jj = 0; jj < J; ++jj) {
    acc[jj] = 0.f;
    const int idx = j0 + jj;
    const bool in = idx < U;
    wr[jj] = in ? rR[(size_t)idx * rs] : 0.f;
    wy[jj] = (!SQ && in) ? yR[(size_t)idx * rs] : 0.f;
  }
  for (int k = 0; k < U; ++k) {
    const float yf = yF[(size_t)k * rs];
    const float rf = SQ ? 0.f : rF[(size_t)k * rs];
#pragma unroll
    for (int jj = 0; jj < J; ++jj) {
      acc[jj] = fmaf(yf, wr[jj], acc[jj]);
      if constexpr (!SQ) acc[jj] = fmaf(rf, wy[jj], acc[jj]);
    }
#pragma unroll
    for (int jj = J - 1; jj > 0; --jj) {
      wr[jj] = wr[jj - 1];
      if constexpr (!SQ) wy[jj] = wy[jj - 1];
    }
    const int idx = j0 - k - 1;  // enters the window at jj = 0 for k+1
    const bool in = idx >= 0 && idx < U;
    wr[0] = in ? rR[(size_t)idx * rs] : 0.f;
    if constexpr (!SQ) wy[0] = in ? yR[(size_t)idx * rs] : 0.f;
  }
  float* dst = ycol + (size_t)(d0 + j0) * rs;
#pragma unroll
  for (int jj = 0; jj < J; ++jj)
    if (j0 + jj < dlen) dst[(size_t)jj * rs] += acc[jj];
}

// The same tile for a side UT known at compile time: every value it reads --
// the two fixed blocks and the window j0-UT+1 .. j0+J-1 of the two recent
// blocks -- is loaded before the first product (one memory round trip, rows
// clamped into range and zero-selected, since a load under a condition would
// wait for the earlier ones), and the window offsets become register names.
template <int J, int UT, bool SQ>
__global__ __launch_bounds__(kThreads) void k_dd_direct_u(float* __restrict__ Y,
                                                          const float* __restrict__ R, int L,
                                                          int BD, int lo, int d0, int dlen) {
  constexpr int NW = J + UT - 1;  // window: recent index j0 - UT + 1 + i, i < NW
  const int c = (int)blockIdx.x * kThreads + (int)threadIdx.x;
  const int j0 = (int)blockIdx.y * J;
  const int m = (int)blockIdx.z;
  if (c >= BD || j0 >= dlen) return;
  const size_t rs = (size_t)BD;
  float* ycol = Y + (size_t)m * L * BD + c;
  const float* rcol = R + (size_t)m * L * BD + c;
  const float* yR = ycol + (size_t)lo * rs;
  const float* rR = rcol + (size_t)lo * rs;
  const float* yF = ycol + (size_t)UT * rs;
  const float* rF = rcol + (size_t)UT * rs;
  float fy[UT], fr[UT], wy[NW], wr[NW];
#pragma unroll
  for (int k = 0; k < UT; ++k) {
    fy[k] = yF[(size_t)k * rs];
    fr[k] = SQ ? 0.f : rF[(size_t)k * rs];
  }
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const int idx = j0 - UT + 1 + i;
    const int cl = idx < 0 ? 0 : (idx >= UT ? UT - 1 : idx);
    const float vr = rR[(size_t)cl * rs];
    const float vy = SQ ? 0.f : yR[(size_t)cl * rs];
    const bool in = idx >= 0 && idx < UT;
    wr[i] = in ? vr : 0.f;
    wy[i] = in ? vy : 0.f;
  }
  float* dst = ycol + (size_t)(d0 + j0) * rs;
#pragma unroll
  for (int jj = 0; jj < J; ++jj) {
    float a = 0.f;
#pragma unroll
    for (int k = 0; k < UT; ++k) {
      a = fmaf(fy[k], wr[jj - k + UT - 1], a);
      if constexpr (!SQ) a = fmaf(fr[k], wy[jj - k + UT - 1], a);
    }
    if (j0 + jj < dlen) dst[(size_t)jj * rs] += a;
  }
}

// ---- FFT parallelogram tiles (2U-point, one LDS-resident pass)
//
// Each real column carries its two blocks packed as one complex signal,
// x = y + i rho (zero-padded to N = 2U).  From X = DFT(x) the spectra of the
// parts follow by conjugate symmetry: Y[k] = (X[k] + conj X[N-k]) / 2,
// Rho[k] = (X[k] - conj X[N-k]) / 2i.  The product spectrum of a column is
// P = YF RhoR + RhoF YR (rectangle; the fixed block F, the recent block R) or
// YF RhoF (square), Hermitian since the output is real, so two columns a, b
// share one inverse: Q = Pa + i Pb, out_a + i out_b = IDFT(Q).  The 2U-1
// outputs of the untruncated convolution are below N, so nothing wraps.
// Per column: 2 forward transforms (1 for the square) and half an inverse.
//
// Launch shape: CW real columns per workgroup (the forward transforms run on
// CW complex columns, the inverse on CW/2), the LDS buffer N x CW complex;
// NT threads.
template <int N>
struct DdCfg {
  static constexpr int CW = N <= 1024 ? 16 : (N <= 2048 ? 8 : (N <= 4096 ? 4 : 2));
  // at most 512 threads: the spectra held across the second transform need
  // more than the 128 registers a 1024-thread workgroup leaves
  static constexpr int NT = N <= 64 ? 64 : (N <= 128 ? 128 : (N <= 256 ? 256 : 512));
  static constexpr bool TWL = (size_t)N * 8 * (CW + 1) <= 163840;
  static constexpr bool TWH = !TWL && (size_t)N * 8 * CW + (size_t)N * 4 <= 163840;
  static constexpr int TWN = TWL ? N : (TWH ? N / 2 : 1);
};

template <int N>
using DdTw = typename std::conditional<
    DdCfg<N>::TWL, fft::TwLds<N>,
    typename std::conditional<DdCfg<N>::TWH, fft::TwLdsHalf<N>, fft::TwGlobal>::type>::type;

template <int N, int NT>
__device__ __forceinline__ DdTw<N> dd_make_tw(float2* lds, const float2* __restrict__ tw) {
  if constexpr (DdCfg<N>::TWL) {
    fft::load_twiddles<N, NT>(lds, tw);
    return fft::TwLds<N>{lds};
  } else if constexpr (DdCfg<N>::TWH) {
    fft::load_twiddles<N, NT, N / 2>(lds, tw);
    return fft::TwLdsHalf<N>{lds};
  } else {
    return fft::TwGlobal{tw};
  }
}

// The two packed parts of X at bin k: (first, second) spectra.
__device__ __forceinline__ void unpack(float2 xk, float2 xnk, float2& a, float2& b) {
  const float2 c = conjf2(xnk);
  a = make_float2(0.5f * (xk.x + c.x), 0.5f * (xk.y + c.y));
  const float2 d = csub(xk, c);  // 2i * b
  b = make_float2(0.5f * d.y, -0.5f * d.x);
}

//
// Tiles wider than the largest single-pass transform (U = K V, V = N / 2)
// are split into V-blocks: fixed sub-blocks F_p = [fo + pV, fo + (p+1)V),
// recent ones R_q = [lo + qV, ...), p, q < K.  The pair (p, q) contributes
// its V-block convolution at offset (p + q) V of the destination, so output
// block r = p + q (rows d0 + rV + j, j < 2V - 1) takes the sum over p of
// the pairs' product spectra -- accumulated in registers, one inverse per r.
// The square sums yF_p (*) rhoF_q over every ordered (p, q); the rectangle
// yF_p (*) rhoR_q + rhoF_p (*) yR_q.  Blocks r and r + 1 overlap by V - 1
// rows, so one launch (MB) covers every other r: r = r0 + 2 j.  K = 1 is
// the plain tile (fo = U).
// Threads of a workgroup: the block-split form keeps a third spectrum (the
// running sum) in registers, so from N = 2048 on it takes 1024 threads.
template <int N, bool MB>
constexpr int dd_threads() {
  return MB && N >= 2048 ? 1024 : DdCfg<N>::NT;
}

template <int N, bool SQ, bool MB>
__global__ __launch_bounds__((dd_threads<N, MB>())) void k_dd_fft(float* __restrict__ Y,
                                                        const float* __restrict__ R,
                                                        const float2* __restrict__ tw, int L,
                                                        int BD, int fo, int lo, int d0, int dlen,
                                                        int ppl, int lm, int K, int r0) {
  constexpr int CW = DdCfg<N>::CW, NT = dd_threads<N, MB>(), U = N / 2, HW = CW / 2;
  __shared__ float2 buf[N * CW];
  __shared__ float2 twl[DdCfg<N>::TWN];
  const auto twz = dd_make_tw<N, NT>(twl, tw);
  const int q = fft::xcd_logical((int)blockIdx.x, (int)gridDim.x);
  const int units = ppl * lm;  // (layer, panel) units per output block
  const int rb = MB ? q / units : 0;
  const int qu = MB ? q - rb * units : q;
  const int m = qu / ppl;
  const int c0 = (qu - m * ppl) * CW;
  const size_t rs = (size_t)BD;
  float* Ym = Y + (size_t)m * L * BD;
  const float* Rm = R + (size_t)m * L * BD;

  constexpr int PUN = (U + 1) * CW;  // (bin kk <= U, column col) units
  constexpr int PU = (PUN + NT - 1) / NT;
  constexpr float inv_n = 1.0f / (float)N;
  // the forward transform of the packed block y + i rho at rows base ..
  // base + U - 1 of the unit's columns, into buf
  auto forward_block = [&](int base) {
    fft::forward_from_global<N, CW, CW, NT, true>(buf, twz, [&](int row, int col) {
      const int c = c0 + col;
      if (c >= BD) return make_float2(0.f, 0.f);
      const size_t e = (size_t)(base + row) * rs + c;
      return make_float2(Ym[e], Rm[e]);
    });
  };
  const int r = MB ? r0 + 2 * rb : 0;
  const int pmin = MB ? (r - K + 1 > 0 ? r - K + 1 : 0) : 0;
  const int pmax = MB ? (r < K - 1 ? r : K - 1) : 0;
  float2 p[PU];  // product spectrum of the unit's column, scaled by 1/N
#pragma unroll
  for (int a = 0; a < PU; ++a) p[a] = make_float2(0.f, 0.f);
  for (int pb = pmin; pb <= pmax; ++pb) {
    const int qb = r - pb;
    if (pb > pmin) __syncthreads();  // the previous pair's spectra have been read
    // spectra of the fixed (sub-)block
    forward_block(fo + pb * U);
    float2 yf[PU], rf[PU];
#pragma unroll
    for (int a = 0; a < PU; ++a) {
      const int u = (int)threadIdx.x + a * NT;
      yf[a] = rf[a] = make_float2(0.f, 0.f);
      if (PUN % NT == 0 || u < PUN) {
        const int kk = u / CW, col = u - kk * CW;
        const int nk = (N - kk) & (N - 1);
        unpack(buf[kk * CW + col], buf[nk * CW + col], yf[a], rf[a]);
      }
    }
    if (SQ && pb == qb) {
#pragma unroll
      for (int a = 0; a < PU; ++a) {
        const float2 v = cmul(yf[a], rf[a]);
        p[a].x = fmaf(v.x, inv_n, p[a].x);
        p[a].y = fmaf(v.y, inv_n, p[a].y);
      }
    } else {
      __syncthreads();  // every unit has read the fixed spectra
      forward_block((SQ ? fo : lo) + qb * U);
#pragma unroll
      for (int a = 0; a < PU; ++a) {
        const int u = (int)threadIdx.x + a * NT;
        if (PUN % NT == 0 || u < PUN) {
          const int kk = u / CW, col = u - kk * CW;
          const int nk = (N - kk) & (N - 1);
          float2 yr, rr;
          unpack(buf[kk * CW + col], buf[nk * CW + col], yr, rr);
          const float2 v = SQ ? cmul(yf[a], rr) : cadd(cmul(yf[a], rr), cmul(rf[a], yr));
          p[a].x = fmaf(v.x, inv_n, p[a].x);
          p[a].y = fmaf(v.y, inv_n, p[a].y);
        }
      }
    }
  }
  // half spectra P[kk][col], kk <= U, into LDS; then the packed inverse
  // input Q of every column pair over the whole buffer (after a barrier:
  // the two layouts overlap)
  __syncthreads();
#pragma unroll
  for (int a = 0; a < PU; ++a) {
    const int u = (int)threadIdx.x + a * NT;
    if (PUN % NT == 0 || u < PUN) buf[u] = p[a];  // u = kk * CW + col
  }
  __syncthreads();
  constexpr int QUN = (U + 1) * HW;
  constexpr int QU = (QUN + NT - 1) / NT;
  float2 qk[QU], qnk[QU];
#pragma unroll
  for (int a = 0; a < QU; ++a) {
    const int u = (int)threadIdx.x + a * NT;
    if (QUN % NT == 0 || u < QUN) {
      const int kk = u / HW, pr = u - kk * HW;
      const float2 pa = buf[kk * CW + 2 * pr], pb = buf[kk * CW + 2 * pr + 1];
      qk[a] = make_float2(pa.x - pb.y, pa.y + pb.x);     // Pa + i Pb
      qnk[a] = make_float2(pa.x + pb.y, pb.x - pa.y);    // conj Pa + i conj Pb
    }
  }
  __syncthreads();
#pragma unroll
  for (int a = 0; a < QU; ++a) {
    const int u = (int)threadIdx.x + a * NT;
    if (QUN % NT == 0 || u < QUN) {
      const int kk = u / HW, pr = u - kk * HW;
      const int nk = (N - kk) & (N - 1);
      buf[kk * HW + pr] = qk[a];
      if (nk != kk) buf[nk * HW + pr] = qnk[a];
    }
  }
  __syncthreads();
  // rows of output block r inside the destination (its linear convolution
  // has N - 1 rows; row N - 1 of the inverse is zero up to rounding)
  const int rlen = dlen - r * U < N - 1 ? dlen - r * U : N - 1;
  fft::inverse_to_global<N, HW, HW, NT, false>(buf, twz, [&](int row, int pr, float2 v) {
    if (row >= rlen) return;
    const int c = c0 + 2 * pr;
    float* dst = Ym + (size_t)(d0 + r * U + row) * rs;
    if (c < BD) dst[c] += v.x;
    if (c + 1 < BD) dst[c + 1] += v.y;
  });
}

}  // namespace
}  // namespace lcsm

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

bool is_pow2(int v) { return v > 0 && (v & (v - 1)) == 0; }

struct DdOptions {
  int direct_max_u;
  int fft_max_n;
};

// Largest tile side of a length-L run: the largest power of two U with
// 2U < L (the square of t+1 = 2U writes from position 2U on; a rectangle
// needs t+1 >= 3U), 0 if none.
int largest_u(int L) {
  int U = 0;
  for (int u = 1; 2 * u < L; u *= 2) U = u;
  return U;
}

int resolve(int M, int B, int D, int L, const lcsm_options* o, DdOptions* r) {
  size_t dummy = 0;
  int e = lcsm_workspace_bytes(M, B, D, L, nullptr, &dummy);  // the common shape checks
  if (e) return e;
  r->direct_max_u = lcsm::kDdDefaultDirectMaxU;
  r->fft_max_n = lcsm::kMaxLdsFftN;
  if (o) {
    for (int k = 0; k < 2; ++k)
      if (o->reserved[k] != 0) return LCSM_EINVAL;
    if (o->scratch_mib != 0 || o->half_state != 0 || o->col_fft_min_n != 0 ||
        o->col_tile_form != 0)
      return LCSM_EINVAL;
    if (o->direct_max_u < 0 || o->lds_fft_max_n < 0) return LCSM_EINVAL;
    if (o->direct_max_u) {
      if (!is_pow2(o->direct_max_u)) return LCSM_EINVAL;
      r->direct_max_u = o->direct_max_u;
    }
    if (o->lds_fft_max_n) {
      if (!is_pow2(o->lds_fft_max_n) || o->lds_fft_max_n < lcsm::kMinLdsFftN ||
          o->lds_fft_max_n > lcsm::kMaxLdsFftN)
        return LCSM_EINVAL;
      r->fft_max_n = o->lds_fft_max_n;
    }
  }
  return LCSM_OK;
}

// Largest FFT length of a context (0: every tile direct): 2U of its largest
// FFT tile, capped at the single-pass limit (wider tiles run as V-blocks).
int fft_nmax(int L, const DdOptions& o) {
  const int Umax = largest_u(L);
  if (Umax <= o.direct_max_u) return 0;
  return 2 * Umax < o.fft_max_n ? 2 * Umax : o.fft_max_n;
}

size_t state_bytes(int M, int B, int D, int L) {
  return align_up(sizeof(float) * (size_t)M * L * B * D);
}

size_t dd_bytes(int M, int B, int D, int L, const DdOptions& o) {
  return 2 * state_bytes(M, B, D, L) + align_up(sizeof(float2) * 2 * (size_t)fft_nmax(L, o));
}

}  // namespace

struct lcsm_dd {
  int M, B, D, L, BD;
  DdOptions opt;
  hipStream_t stream;
  bool owns_ws;
  char* ws;
  float* Y;
  float* R;
  float2* tw;  // twiddles of the FFT tiles (nullptr: every tile direct)
  int t;
  bool faulted;
  char msg[256];
};

namespace {

int dd_fail(lcsm_dd* c, int code, const char* what, hipError_t e) {
  if (e != hipSuccess) {
    snprintf(c->msg, sizeof(c->msg), "%s: %s", what, hipGetErrorString(e));
    c->faulted = true;
    return LCSM_EDEVICE;
  }
  snprintf(c->msg, sizeof(c->msg), "%s", what);
  return code;
}

// The FFT tile of side U for all layers: one 2U-point launch when 2U fits
// the single-pass limit, else V-blocks (V = fft_max_n / 2, K = U / V) in two
// launches, the even and then the odd output blocks r < 2K - 1 that start
// inside the destination.
template <bool SQ>
hipError_t dd_fft(lcsm_dd* c, int U, int lo, int d0, int dlen) {
  const int N = 2 * U <= c->opt.fft_max_n ? 2 * U : c->opt.fft_max_n;
  const int V = N / 2, K = U / V;
  // output blocks that start inside the destination (r V < dlen), at most 2K - 1
  const int nb = (dlen + V - 1) / V < 2 * K - 1 ? (dlen + V - 1) / V : 2 * K - 1;
#define LCSM_CASE(NN)                                                                             \
  case NN: {                                                                                      \
    constexpr int CW = lcsm::DdCfg<NN>::CW;                                                       \
    const int ppl = (c->BD + CW - 1) / CW;                                                        \
    if (K == 1) {                                                                                 \
      hipLaunchKernelGGL((lcsm::k_dd_fft<NN, SQ, false>), dim3((unsigned)(ppl * c->M)),           \
                         dim3(lcsm::DdCfg<NN>::NT), 0, c->stream, c->Y, c->R, c->tw, c->L, c->BD, \
                         U, lo, d0, dlen, ppl, c->M, 1, 0);                                       \
      return hipGetLastError();                                                                   \
    }                                                                                             \
    for (int r0 = 0; r0 < 2 && r0 < nb; ++r0) {                                                   \
      const int nr = (nb - r0 + 1) / 2;                                                           \
      hipLaunchKernelGGL((lcsm::k_dd_fft<NN, SQ, true>), dim3((unsigned)(nr * ppl * c->M)),       \
                         dim3(lcsm::dd_threads<NN, true>()), 0, c->stream, c->Y, c->R, c->tw, c->L, c->BD, \
                         U, lo, d0, dlen, ppl, c->M, K, r0);                                      \
      const hipError_t e = hipGetLastError();                                                     \
      if (e != hipSuccess) return e;                                                              \
    }                                                                                             \
    return hipSuccess;                                                                            \
  }
  switch (N) {
    LCSM_CASE(4)
    LCSM_CASE(8)
    LCSM_CASE(16)
    LCSM_CASE(32)
    LCSM_CASE(64)
    LCSM_CASE(128)
    LCSM_CASE(256)
    LCSM_CASE(512)
    LCSM_CASE(1024)
    LCSM_CASE(2048)
    LCSM_CASE(4096)
    LCSM_CASE(8192)
  }
#undef LCSM_CASE
  return hipErrorInvalidValue;
}

// One tile of side U for all layers: direct up to the crossover, else the
// 2U-point FFT tile.
hipError_t dd_tile(lcsm_dd* c, bool square, int U, int lo, int d0, int dlen) {
  if (U > c->opt.direct_max_u)
    return square ? dd_fft<true>(c, U, lo, d0, dlen) : dd_fft<false>(c, U, lo, d0, dlen);
  const dim3 grid((unsigned)((c->BD + lcsm::kThreads - 1) / lcsm::kThreads),
                  (unsigned)((dlen + lcsm::kDdJ - 1) / lcsm::kDdJ), (unsigned)c->M);
#define LCSM_DD_U(UU)                                                                              \
  if (U == UU) {                                                                                   \
    if (square)                                                                                    \
      hipLaunchKernelGGL((lcsm::k_dd_direct_u<lcsm::kDdJ, UU, true>), grid, dim3(lcsm::kThreads), 0, \
                         c->stream, c->Y, c->R, c->L, c->BD, lo, d0, dlen);                        \
    else                                                                                           \
      hipLaunchKernelGGL((lcsm::k_dd_direct_u<lcsm::kDdJ, UU, false>), grid, dim3(lcsm::kThreads),   \
                         0, c->stream, c->Y, c->R, c->L, c->BD, lo, d0, dlen);                     \
    return hipGetLastError();                                                                      \
  }
  LCSM_DD_U(16)
  LCSM_DD_U(32)
#undef LCSM_DD_U
  if (square)
    hipLaunchKernelGGL((lcsm::k_dd_direct<lcsm::kDdJ, true>), grid, dim3(lcsm::kThreads), 0,
                       c->stream, c->Y, c->R, c->L, c->BD, U, lo, d0, dlen);
  else
    hipLaunchKernelGGL((lcsm::k_dd_direct<lcsm::kDdJ, false>), grid, dim3(lcsm::kThreads), 0,
                       c->stream, c->Y, c->R, c->L, c->BD, U, lo, d0, dlen);
  return hipGetLastError();
}

}  // namespace

extern "C" {

int lcsm_dd_workspace_bytes(int M, int B, int D, int L, const lcsm_options* opt, size_t* bytes) {
  if (!bytes) return LCSM_EINVAL;
  DdOptions o;
  int r = resolve(M, B, D, L, opt, &o);
  if (r) return r;
  *bytes = dd_bytes(M, B, D, L, o);
  return LCSM_OK;
}

int lcsm_dd_init(lcsm_dd** out, int M, int B, int D, int L, void* stream, void* workspace,
                 size_t workspace_bytes, const lcsm_options* opt) {
  if (!out) return LCSM_EINVAL;
  *out = nullptr;
  DdOptions o;
  int r = resolve(M, B, D, L, opt, &o);
  if (r) return r;
  const size_t need = dd_bytes(M, B, D, L, o);
  if (workspace) {
    if (workspace_bytes < need) return LCSM_ENOMEM;
    if (((uintptr_t)workspace) % kAlign) return LCSM_EINVAL;
  }
  lcsm_dd* c = new (std::nothrow) lcsm_dd();
  if (!c) return LCSM_ENOMEM;
  c->M = M;
  c->B = B;
  c->D = D;
  c->L = L;
  c->BD = B * D;
  c->opt = o;
  c->stream = (hipStream_t)stream;
  c->msg[0] = 0;
  if (workspace) {
    c->ws = (char*)workspace;
    c->owns_ws = false;
  } else {
    void* p = nullptr;
    if (hipMalloc(&p, need) != hipSuccess) {
      (void)hipGetLastError();
      delete c;
      return LCSM_ENOMEM;
    }
    c->ws = (char*)p;
    c->owns_ws = true;
  }
  const size_t sb = state_bytes(M, B, D, L);
  c->Y = (float*)c->ws;
  c->R = (float*)(c->ws + sb);
  const int nmax = fft_nmax(L, o);
  c->tw = nmax ? (float2*)(c->ws + 2 * sb) : nullptr;
  hipError_t e = lcsm::launch_zero((float*)c->ws, 2 * sb / sizeof(float), c->stream);
  if (e == hipSuccess && nmax) {
    std::vector<float2> t = lcsm::twiddle_table(nmax);
    e = hipMemcpyAsync(c->tw, t.data(), t.size() * sizeof(float2), hipMemcpyHostToDevice,
                       c->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(c->stream);  // the host table must outlive the copy
  }
  if (e != hipSuccess) {
    (void)hipGetLastError();
    if (c->owns_ws) (void)hipFree(c->ws);
    delete c;
    return LCSM_EDEVICE;
  }
  c->t = 0;
  c->faulted = false;
  *out = c;
  return LCSM_OK;
}

int lcsm_dd_step(lcsm_dd* c, const float* y_t, const float* rho_t, float* z_t) {
  if (!c) return LCSM_EINVAL;
  if (!y_t || !rho_t || !z_t)
    return dd_fail(c, LCSM_EINVAL, "null input or output pointer", hipSuccess);
  if (c->faulted) return LCSM_ESTATE;
  if (c->t >= c->L) return LCSM_EDONE;
  const int t = c->t;
  // every power of two U dividing t+1 with 2U <= t+1: those up to the fused
  // limit (and the direct limit) go with the red cell, the rest one launch
  // per U
  const int i1 = t + 1;
  const int fmax = c->opt.direct_max_u < lcsm::kDdFusedMaxU ? c->opt.direct_max_u
                                                            : lcsm::kDdFusedMaxU;
  int uf = 0;
  for (int U = 1; U <= fmax && i1 % U == 0 && 2 * U <= i1; U *= 2) uf = U;
  const dim3 rgrid((unsigned)((c->BD + lcsm::kThreads - 1) / lcsm::kThreads), (unsigned)c->M);
#define LCSM_DD_STEP(UU)                                                                        \
  hipLaunchKernelGGL((lcsm::k_dd_step<UU>), rgrid, dim3(lcsm::kThreads), 0, c->stream, y_t,    \
                     rho_t, z_t, c->Y, c->R, c->L, c->BD, t)
  switch (uf) {
    case 0: LCSM_DD_STEP(0); break;
    case 1: LCSM_DD_STEP(1); break;
    case 2: LCSM_DD_STEP(2); break;
    case 4: LCSM_DD_STEP(4); break;
    default: LCSM_DD_STEP(8); break;
  }
#undef LCSM_DD_STEP
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return dd_fail(c, LCSM_EDEVICE, "red-cell launch", e);
  for (int U = 2 * uf > 0 ? 2 * uf : 1; i1 % U == 0 && 2 * U <= i1; U *= 2) {
    const bool square = i1 == 2 * U;
    const int lo = square ? U : t - U + 1;
    const int d0 = square ? 2 * U : t + 1;
    if (d0 >= c->L) continue;
    const int dlen = (d0 + 2 * U - 1 <= c->L ? 2 * U - 1 : c->L - d0);
    e = dd_tile(c, square, U, lo, d0, dlen);
    if (e != hipSuccess) return dd_fail(c, LCSM_EDEVICE, "tile launch", e);
  }
  c->t = t + 1;
  return LCSM_OK;
}

int lcsm_dd_reset(lcsm_dd* c) {
  if (!c) return LCSM_EINVAL;
  const size_t n = 2 * state_bytes(c->M, c->B, c->D, c->L) / sizeof(float);
  hipError_t e = lcsm::launch_zero((float*)c->ws, n, c->stream);
  if (e != hipSuccess) return dd_fail(c, LCSM_EDEVICE, "reset", e);
  c->t = 0;
  c->faulted = false;
  c->msg[0] = 0;
  return LCSM_OK;
}

int lcsm_dd_position(const lcsm_dd* c, int* t) {
  if (!c || !t) return LCSM_EINVAL;
  *t = c->t;
  return LCSM_OK;
}

void lcsm_dd_destroy(lcsm_dd* c) {
  if (!c) return;
  (void)hipStreamSynchronize(c->stream);
  if (c->owns_ws) (void)hipFree(c->ws);
  delete c;
}

const char* lcsm_dd_last_error(const lcsm_dd* c) { return c ? c->msg : ""; }

}  // extern "C"
