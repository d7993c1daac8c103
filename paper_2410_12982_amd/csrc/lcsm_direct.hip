// Red cells and direct (Toeplitz) gray tiles of the relaxed online
// convolution, for gfx950.
//
// Layout: state S[m][t][c] with c = b*D + d (time-major, one B*D slab per
// position and layer), filters Hf[m][k][d] (lag-major).  A thread owns one
// column (m, c): every element it writes has no other writer in the launch,
// so results are deterministic and no atomics are used.  Consecutive threads
// take consecutive c, so every row access of a wavefront is one contiguous
// 256-byte segment.
//
// Red cell (Alg. 1 red line, Alg. 3 inner loop): z_t = fmaf(h_0, y_t, acc_t),
// then the slot of position t is overwritten with y_t (the in-place storage
// of Sec. 3.3: b^l_t lives in a^l_t's slot until it is consumed).
//
// Gray tile (Eq. taus) for i = t+1, side U: for j < dst_len,
//   S[i+j] += sum_{k<U} y[i-U+k] * h[U+j-k]     (lags 1..2U-1).
#include <type_traits>
#include <utility>

#include "lcsm_internal.h"

namespace lcsm {
namespace {

constexpr int kThreads = 256;

// Output split of the fused tile: SPLIT threads share one column, each
// computing U/SPLIT of the U outputs (bounds the per-thread work and
// registers at the larger fused sides).
template <int U>
struct Split {
  static constexpr int value = U >= 64 ? 8 : (U >= 32 ? 4 : (U >= 16 ? 2 : 1));
};

// RED: do the red cell at position t first (the tile's newest input y_t then
// comes from the register, not from memory).  U == 0: no tile.
// 1 <= U <= kFusedMaxU: the tile i = t+1 (U outputs from U inputs and 2U-1
// lags) is computed by SPLIT threads per column, thread part p taking the
// outputs j in [p U/SPLIT, (p+1) U/SPLIT); part 0 also does the red cell.
// Every load (inputs, lags, the red cell's accumulator and the tile's
// destination accumulators) is issued before the first store, so the step
// costs one memory round trip; the slots read and written are distinct rows.
// Grid (channel blocks, B, M * SPLIT): no integer division on the critical
// path, consecutive lanes take consecutive channels.  With a channel-block
// count that is not a multiple of 8 the batch rows of one block run on
// different XCDs, and each XCD's L2 fetches the same lag rows.  Remapping the
// workgroup ids so that they share one XCD removes those reads, but its
// integer divisions ahead of the first load cost about 0.5 us per launch on
// these latency-bound steps (a 32768-position, 18-layer generation: 135 ->
// 151 ms), so the grid keeps the hardware order.
template <int U, bool RED>
__global__ __launch_bounds__(kThreads) void k_step_fused(const float* __restrict__ y,
                                                        float* __restrict__ z,
                                                        float* __restrict__ S,
                                                        const float* __restrict__ Hf, int m0, int L,
                                                        int SL, int BD, int D, int t, int dst_len) {
  constexpr int SP = U > 0 ? Split<U>::value : 1;
  constexpr int UJ = U > 0 ? U / SP : 1;  // outputs per thread
  const int d = (int)blockIdx.x * kThreads + (int)threadIdx.x;
  if (d >= D) return;
  const int m = m0 + (int)blockIdx.z / SP;
  const int part = (int)blockIdx.z - (m - m0) * SP;
  const int j0 = part * UJ;
  const int c = (int)blockIdx.y * D + d;
  const size_t e = (size_t)m * BD + c;
  float* col = S + (size_t)m * SL * BD + c;
  const float* hc = Hf + (size_t)m * L * D + d;
  const size_t rs = (size_t)BD;

  constexpr int NY = U > 0 ? U : 1;
  constexpr int NH = U > 0 ? UJ + U : 1;  // lags j0+1 .. j0+UJ+U-1 at hh[1..]
  float yb[NY];
  float hh[NH];
  float zo[UJ];
  const bool tile = (U > 0) && (j0 < dst_len);
  const bool red = RED && part == 0;
  // Every load is unconditional, with its row or lag clamped into range
  // (values past the end are never used): loads under a condition are issued
  // only after the earlier ones have returned, a second round trip per step.
  float yt, acc = 0.f, h0 = 0.f;
  if constexpr (RED) {
    yt = y[e];
    acc = col[(size_t)t * rs];
    h0 = hc[0];
  } else {
    yt = col[(size_t)t * rs];
  }
  if constexpr (U > 0) {
    // rows t+1-U .. t-1 already hold inputs (U divides t+1); row t is y_t
#pragma unroll
    for (int k = 0; k < U - 1; ++k) yb[k] = col[(size_t)(t + 1 - U + k) * rs];
    // output j uses lags U+j-k, k < U: for j in [j0, j0+UJ) that is j0+1 .. j0+UJ+U-1
#pragma unroll
    for (int l = 1; l < UJ + U; ++l) {
      const int lag = j0 + l;
      const float v = hc[(size_t)(lag < L ? lag : L - 1) * D];
      hh[l] = lag < L ? v : 0.f;
    }
#pragma unroll
    for (int jj = 0; jj < UJ; ++jj) {
      const int row = t + 1 + j0 + jj;
      zo[jj] = col[(size_t)(row < L ? row : L - 1) * rs];
    }
  }
  // Pin every loaded value here, after the last load (an empty statement
  // that reads and writes each register): no load is sunk into the
  // conditional red-cell or tile blocks below, and all of them are in flight
  // together.  The tile's values only up to U = 16: with the 80 and more
  // values of the larger tiles held at once the compiler issues the loads in
  // small groups instead.
  constexpr bool PIN = U <= 16;
  // y_t as well without the red cell: with nothing pinned there, the tile of
  // U = 32 issued its lag loads one round trip each
  if constexpr (RED)
    asm volatile("" : "+v"(acc), "+v"(h0));
  else
    asm volatile("" : "+v"(yt));
  if constexpr (U > 0 && PIN) {
#pragma unroll
    for (int l = 1; l < UJ + U; ++l) asm volatile("" : "+v"(hh[l]));
#pragma unroll
    for (int jj = 0; jj < UJ; ++jj) asm volatile("" : "+v"(zo[jj]));
#pragma unroll
    for (int k = 0; k < U - 1; ++k) asm volatile("" : "+v"(yb[k]));
  }
  if (red) {
    z[e] = fmaf(h0, yt, acc);
    col[(size_t)t * rs] = yt;
  }
  if constexpr (U > 0) {
    if (tile) {
      yb[U - 1] = yt;
#pragma unroll
      for (int jj = 0; jj < UJ; ++jj) {
        if (j0 + jj < dst_len) {
          float o = 0.f;
#pragma unroll
          for (int k = 0; k < U; ++k) o = fmaf(yb[k], hh[U + jj - k], o);
          col[(size_t)(t + 1 + j0 + jj) * rs] = zo[jj] + o;
        }
      }
    }
  }
}

// The chain's input rule y = x + 0.5 tanh(z), evaluated as
// (x + 1/2) - 1/(1 + e^{2z}) (the same function: 0.5 tanh(z) = 1/2 -
// 1/(1 + e^{2z})) from the hardware base-2 exponential and reciprocal (each
// within about one ulp): no branch, and x + 1/2 is off the serial chain.
// Absolute error below 3.3e-7 for |x| <= 3 (an fp32 model of these steps
// with both hardware results off by one ulp either way, against fp64, on
// 1.2M points with z over [-20, 20] and 1e-8 .. 32 of either sign); z = +inf
// gives x + 1/2, z = -inf x - 1/2, NaN stays NaN.
__device__ __forceinline__ float chain_y(float x, float z) {
  const float e = __builtin_amdgcn_exp2f(2.8853900817779268f * z);  // e^{2z}
  return (x + 0.5f) - __builtin_amdgcn_rcpf(1.f + e);
}

template <int U>
struct ChainChunk {
  static constexpr int value = U <= 2 ? 8 : (U <= 8 ? 4 : (U <= 16 ? 2 : 1));
};

template <int U, int K>
__global__ __launch_bounds__(kThreads) void k_chain_fused(const float* __restrict__ x,
                                                         float* __restrict__ z,
                                                         float* __restrict__ S,
                                                         const float* __restrict__ Hf,
                                                         float* __restrict__ prev, int M, int L,
                                                         int SL, int BD, int D, int t,
                                                         int dst_len) {
  constexpr int NY = U > 0 ? U : 1;
  constexpr int NH = U > 0 ? 2 * U : 1;
  constexpr int NZ = U > 0 ? U : 1;
  const int d = (int)blockIdx.x * kThreads + (int)threadIdx.x;
  if (d >= D) return;
  const int c = (int)blockIdx.y * D + d;
  const size_t rs = (size_t)BD;
  const bool tile = (U > 0) && (dst_len > 0);
  float zl = 0.f;  // z^{M-1}_{t-1} (loaded with the first chunk), then z^{m-1}_t
  for (int m0 = 0; m0 < M; m0 += K) {
    float xv[K], acc[K], h0[K];
    float yb[K][NY], hh[K][NH], zo[K][NZ];
    // loads of the chunk's layers (past the last layer: layer M-1 again,
    // unused; rows and lags clamped into range)
#pragma unroll
    for (int kk = 0; kk < K; ++kk) {
      const int m = m0 + kk < M ? m0 + kk : M - 1;
      const float* col = S + (size_t)m * SL * BD + c;
      const float* hc = Hf + (size_t)m * L * D + d;
      xv[kk] = x[(size_t)m * BD + c];
      acc[kk] = col[(size_t)t * rs];
      h0[kk] = hc[0];
      if constexpr (U > 0) {
#pragma unroll
        for (int k = 0; k < U - 1; ++k) yb[kk][k] = col[(size_t)(t + 1 - U + k) * rs];
#pragma unroll
        for (int l = 1; l < 2 * U; ++l) {
          const float v = hc[(size_t)(l < L ? l : L - 1) * D];
          hh[kk][l] = l < L ? v : 0.f;
        }
#pragma unroll
        for (int j = 0; j < U; ++j) {
          const int row = t + 1 + j;
          zo[kk][j] = col[(size_t)(row < L ? row : L - 1) * rs];
        }
      }
    }
    if (m0 == 0) zl = prev[c];  // unused at t = 0
    // the chain through the chunk, then its stores
#pragma unroll
    for (int kk = 0; kk < K; ++kk) {
      const int m = m0 + kk;
      if (m < M) {
        float* col = S + (size_t)m * SL * BD + c;
        const float yv = (m == 0 && t == 0) ? xv[kk] : chain_y(xv[kk], zl);
        const float zv = fmaf(h0[kk], yv, acc[kk]);
        z[(size_t)m * BD + c] = zv;
        col[(size_t)t * rs] = yv;
        zl = zv;
        if constexpr (U > 0) {
          if (tile) {
            yb[kk][U - 1] = yv;
#pragma unroll
            for (int j = 0; j < U; ++j) {
              if (j < dst_len) {
                float o = 0.f;
#pragma unroll
                for (int k = 0; k < U; ++k) o = fmaf(yb[kk][k], hh[kk][U + j - k], o);
                col[(size_t)(t + 1 + j) * rs] = zo[kk][j] + o;
              }
            }
          }
        }
      }
    }
  }
  prev[c] = zl;
}

// The chained steps (lcsm_step_chain) of the positions [t0, t1) of one
// aligned block of kChainBlockW positions (b = t0 rounded down to it), in
// one launch, when every gray tile of the stretch is direct with
// U <= kChainBlockW / 2 (the tile of the last position only when
// tile_last).  Such a tile, of i = b + r + 1 with r + 1 < kChainBlockW,
// reads y rows [i - U, i) and adds into rows [i, i + U), all inside
// [b, b + kChainBlockW): the block's rows of a column stay in that column's
// registers from the first position to the last, and no position of the
// stretch moves a tile's operands through memory.
//
// A workgroup owns kChainBlockCols (b, d) columns of every layer.  Wave 0
// walks the chain through the layers (y^m_t, z^m_t as k_chain_fused) on its
// first kChainBlockCols lanes; wave w >= 1 holds layers 2(w-1) and
// 2(w-1)+1, one per half.  Each lane of a layer wave keeps v[k] = state row
// b + k of its column (y for positions already taken, the accumulator
// otherwise) and the lags 1 .. kChainBlockW - 1 of its channel.  Per
// position t = b + r: the layer waves hand acc_t and x_t over in LDS
// (fetching x_{t+1}); wave 0 computes the chain and leaves z_t and y_t in
// LDS, while the layer waves add the other output rows of the previous
// position's tile; then each layer wave stores its layers' z_t and y_t
// (W0S, for at most kChainBlockWave0StoreM layers: wave 0 stores them as
// it goes instead) and computes the first output row of the tile of i = t+1 (the next
// accumulator).  The tile arithmetic is that of k_step_fused<U, false> (per
// output, the fmaf chain over the U inputs in increasing order, then added
// to the accumulator), so the results equal the per-position steps bit for
// bit.  The two barriers per position order LDS only: no wave reads global
// memory another wave of the launch writes.  At the end the accumulator rows
// at and after t1 (a stretch cut before its block ends) go back to the state.

// f(std::integral_constant<int, 0>{}), ..., f(std::integral_constant<int, N-1>{}).
template <class F, int... R>
__device__ __forceinline__ void static_for_impl(F& f, std::integer_sequence<int, R...>) {
  (f(std::integral_constant<int, R>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

__device__ __forceinline__ void chain_block_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// The tile of i = b + R + 1 (U = lowbit(R + 1)) on the register rows v, in
// two parts: its first output row (R + 1, the accumulator the next
// position's chain needs) and the rest (rows R + 2 .. R + U).  rem = L - i
// clips the rows past the end.
template <int R>
__device__ __forceinline__ void chain_block_first_row(float (&v)[kChainBlockW],
                                                      const float (&hh)[kChainBlockW]) {
  constexpr int U = (R + 1) & -(R + 1);
  float o = 0.f;
#pragma unroll
  for (int k = 0; k < U; ++k) o = fmaf(v[R + 1 - U + k], hh[U - k], o);
  v[R + 1] = v[R + 1] + o;
}

template <int R>
__device__ __forceinline__ void chain_block_rest_rows(float (&v)[kChainBlockW],
                                                      const float (&hh)[kChainBlockW], int rem) {
  constexpr int U = (R + 1) & -(R + 1);
#pragma unroll
  for (int j = 1; j < U; ++j) {
    if (j < rem) {
      float o = 0.f;
#pragma unroll
      for (int k = 0; k < U; ++k) o = fmaf(v[R + 1 - U + k], hh[U + j - k], o);
      v[R + 1 + j] = v[R + 1 + j] + o;
    }
  }
}

template <bool W0S>
__global__ __launch_bounds__(64 * (1 + (kChainBlockMaxM + 1) / 2)) void k_chain_block(
    const float* __restrict__ x, size_t xst, int xring, int xs0, float* __restrict__ z,
    size_t zst, int zring, int zs0, float* __restrict__ S, const float* __restrict__ Hf,
    float* __restrict__ prev, int M, int L, int SL, int BD, int D, int t0, int t1,
    int tile_last) {
  constexpr int NC = kChainBlockCols, W = kChainBlockW;
  __shared__ float2 axbuf[kChainBlockMaxM][NC];  // (acc_t, x_t)
  __shared__ float2 yzbuf[kChainBlockMaxM][NC];  // (y_t, z_t)
  __shared__ float h0buf[kChainBlockMaxM][NC];
  const int lane = (int)threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int col = lane & (NC - 1);
  const int c = (int)blockIdx.x * NC + col;
  const bool live = c < BD;
  const int cc = live ? c : BD - 1;
  const int d = cc % D;
  const size_t rs = (size_t)BD;
  const int b = t0 & ~(W - 1);
  const int r0 = t0 - b, r1 = t1 - b;
  const int m = 2 * (wv - 1) + (lane >> 5);
  const bool has = wv > 0 && m < M;
  const int mc = has ? m : 0;
  float* Sc = S + (size_t)mc * SL * BD + cc;
  const float* hc = Hf + (size_t)mc * L * D + d;
  const size_t xoff = (size_t)mc * BD + cc;
  float v[W], hh[W];
  float xn = 0.f;
  if (has) {
#pragma unroll
    for (int k = 0; k < W; ++k) v[k] = Sc[(size_t)(b + k < L ? b + k : L - 1) * rs];
    hh[0] = 0.f;
#pragma unroll
    for (int l = 1; l < W; ++l) {
      const float hv = hc[(size_t)(l < L ? l : L - 1) * D];
      hh[l] = l < L ? hv : 0.f;
    }
    h0buf[m][col] = hc[0];
    xn = x[(size_t)(xs0 % xring) * xst + xoff];
  } else {
#pragma unroll
    for (int k = 0; k < W; ++k) v[k] = hh[k] = 0.f;
  }
  float zl = 0.f;  // chain wave: z^{M-1}_{t-1}, then z^{m-1}_t
  if (wv == 0) zl = prev[cc];  // unused at t = 0
  // whether the tile of position p (i = b + p + 1) runs in this launch
  auto tile_of = [&](int p) {
    return p >= r0 && p < r1 && p + 1 < W && b + p + 1 < L && (p + 1 < r1 || tile_last);
  };
  // ring slabs of the current position's z and of the next position's x
  int zsl = zs0 % zring, xsl = (xs0 + 1) % xring;
  auto position = [&](auto rc) {
    constexpr int r = decltype(rc)::value;
    if (r < r0 || r >= r1) return;
    const int t = b + r;
    if (has) {
      axbuf[m][col] = make_float2(v[r], xn);
      if (r + 1 < r1) xn = x[(size_t)xsl * xst + xoff];
      xsl = xsl + 1 == xring ? 0 : xsl + 1;
    }
    chain_block_sync();
    if (wv == 0) {
      if (lane < NC) {
        float* zq = z + (size_t)zsl * zst + c;
        float* Sq = S + (size_t)t * rs + c;
        const size_t ls = (size_t)SL * BD;
        // layer q's inputs read two layers ahead of the chain
        const int q1 = M > 1 ? 1 : 0;
        float2 ax = axbuf[0][col], ax1 = axbuf[q1][col];
        float h0 = h0buf[0][col], h01 = h0buf[q1][col];
        for (int q = 0; q < M; ++q) {
          const int qn = q + 2 < M ? q + 2 : M - 1;
          const float2 ax2 = axbuf[qn][col];
          const float h02 = h0buf[qn][col];
          const float xv = ax.y, av = ax.x;
          const float yv = (q == 0 && t == 0) ? xv : chain_y(xv, zl);
          const float zv = fmaf(h0, yv, av);
          if constexpr (W0S) {
            if (live) {
              zq[(size_t)q * BD] = zv;
              Sq[(size_t)q * ls] = yv;
            }
          }
          yzbuf[q][col] = make_float2(yv, zv);
          zl = zv;
          ax = ax1;
          h0 = h01;
          ax1 = ax2;
          h01 = h02;
        }
      }
    } else if (has && r >= 1) {
      // the rest of the previous position's tile, beside the chain
      if constexpr (r >= 1) {
        if (tile_of(r - 1)) chain_block_rest_rows<r - 1>(v, hh, L - t);
      }
    }
    chain_block_sync();
    if (has) {
      const float2 yz = yzbuf[m][col];
      const float yv = yz.x;
      if constexpr (!W0S) {
        if (live) {
          z[(size_t)zsl * zst + (size_t)m * BD + c] = yz.y;
          Sc[(size_t)t * rs] = yv;
        }
      }
      v[r] = yv;
      if constexpr (r + 1 < W) {
        if (tile_of(r)) chain_block_first_row<r>(v, hh);
      }
    }
    zsl = zsl + 1 == zring ? 0 : zsl + 1;
  };
  static_for<W>(position);
  // the rest of the last position's tile
  auto last_rest = [&](auto rc) {
    constexpr int r = decltype(rc)::value;
    if constexpr (r + 1 < W) {
      if (r == r1 - 1 && tile_of(r)) chain_block_rest_rows<r>(v, hh, L - (b + r + 1));
    }
  };
  if (has) static_for<W>(last_rest);
  if (wv == 0 && lane < NC && live && r1 > r0) prev[c] = zl;
  if (has && live) {
#pragma unroll
    for (int k = 0; k < W; ++k)
      if (k >= r1 && b + k < L) Sc[(size_t)(b + k) * rs] = v[k];
  }
}

// Red cell of one layer.
__global__ __launch_bounds__(kThreads) void k_red_layer(const float* __restrict__ y,
                                                       float* __restrict__ z,
                                                       float* __restrict__ Sm,
                                                       const float* __restrict__ Hm, int BD, int D,
                                                       int t) {
  const int c = blockIdx.x * kThreads + threadIdx.x;
  if (c >= BD) return;
  float* p = Sm + (size_t)t * BD + c;
  const float yt = y[c];
  z[c] = fmaf(Hm[c % D], yt, *p);
  *p = yt;
}

// Direct gray tile for U >= J (U a multiple of J): thread = (column c,
// output chunk j0 .. j0+J-1, layer m).  The J lags needed at input k form a
// window that slides down by one per k, so each step loads one input and one
// new lag.
template <int J>
__global__ __launch_bounds__(kThreads) void k_direct_tile(float* __restrict__ S,
                                                         const float* __restrict__ Hf, int L,
                                                         int SL, int BD, int D, int i, int U,
                                                         int dst_len) {
  const int c = blockIdx.x * kThreads + threadIdx.x;
  const int j0 = blockIdx.y * J;
  const int m = blockIdx.z;
  if (c >= BD || j0 >= dst_len) return;
  const int d = c % D;
  const size_t rs = (size_t)BD;
  float* col = S + (size_t)m * SL * BD + c;
  const float* hc = Hf + (size_t)m * L * D + d;

  float acc[J];
  float w[J];  // w[jj] = h[U + j0 + jj - k] at input k
#pragma unroll
  for (int jj = 0; jj < J; ++jj) {
    acc[jj] = 0.f;
    const int lag = U + j0 + jj;
    w[jj] = (lag < L) ? hc[(size_t)lag * D] : 0.f;
  }
  const float* ysrc = col + (size_t)(i - U) * rs;
  for (int k = 0; k < U; ++k) {
    const float yk = ysrc[(size_t)k * rs];
#pragma unroll
    for (int jj = 0; jj < J; ++jj) acc[jj] = fmaf(yk, w[jj], acc[jj]);
#pragma unroll
    for (int jj = J - 1; jj > 0; --jj) w[jj] = w[jj - 1];
    const int lag = U + j0 - k - 1;  // >= j0 >= 0
    w[0] = (k + 1 < U) ? hc[(size_t)lag * D] : 0.f;
  }
  float* dst = col + (size_t)(i + j0) * rs;
#pragma unroll
  for (int jj = 0; jj < J; ++jj)
    if (j0 + jj < dst_len) dst[(size_t)jj * rs] += acc[jj];
}

__global__ __launch_bounds__(kThreads) void k_transpose(const float* __restrict__ src,
                                                       float* __restrict__ dst, int D, int L) {
  // src [D][L] -> dst [L][D] for layer blockIdx.z; 32x32 tiles, padded LDS.
  // Channel tiles on x (up to 2^31 blocks), lag tiles on y (L <= 2^19 gives
  // at most 16384, inside the 65536-block limit of y and z).
  __shared__ float tile[32][33];
  const size_t off = (size_t)blockIdx.z * D * L;
  const int d0 = blockIdx.x * 32, l0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
  for (int r = ty; r < 32; r += 8) {
    const int d = d0 + r, l = l0 + tx;
    if (d < D && l < L) tile[r][tx] = src[off + (size_t)d * L + l];
  }
  __syncthreads();
  for (int r = ty; r < 32; r += 8) {
    const int l = l0 + r, d = d0 + tx;
    if (d < D && l < L) dst[off + (size_t)l * D + d] = tile[tx][r];
  }
}

// Prompt rows in: S[m][t][c] = y[t * ys + m * BD + c] for t < P (grid-stride
// over P * M * BD, consecutive threads on consecutive c).
__global__ __launch_bounds__(kThreads) void k_rows_in(const float* __restrict__ y, size_t ys,
                                                     float* __restrict__ S, int M, int SL, int BD,
                                                     int P) {
  const size_t n = (size_t)P * M * BD, stride = (size_t)gridDim.x * kThreads;
  for (size_t e = (size_t)blockIdx.x * kThreads + threadIdx.x; e < n; e += stride) {
    const size_t tm = e / BD;
    const int c = (int)(e - tm * BD);
    const int m = (int)(tm % M), t = (int)(tm / M);
    S[((size_t)m * SL + t) * BD + c] = y[t * ys + (size_t)m * BD + c];
  }
}

// State rows out: z[t * zs + m * BD + c] = S[m][row0 + t][c], then the state
// entry is cleared, for t < P.
__global__ __launch_bounds__(kThreads) void k_rows_out_clear(float* __restrict__ S, int M, int SL,
                                                            int BD, int row0, int P,
                                                            float* __restrict__ z, size_t zs) {
  const size_t n = (size_t)P * M * BD, stride = (size_t)gridDim.x * kThreads;
  for (size_t e = (size_t)blockIdx.x * kThreads + threadIdx.x; e < n; e += stride) {
    const size_t tm = e / BD;
    const int c = (int)(e - tm * BD);
    const int m = (int)(tm % M), t = (int)(tm / M);
    float* p = S + ((size_t)m * SL + row0 + t) * BD + c;
    z[t * zs + (size_t)m * BD + c] = *p;
    *p = 0.f;
  }
}

__global__ __launch_bounds__(kThreads) void k_zero(float* __restrict__ p, size_t n) {
  const size_t stride = (size_t)gridDim.x * kThreads;
  for (size_t k = (size_t)blockIdx.x * kThreads + threadIdx.x; k < n; k += stride) p[k] = 0.f;
}

// Zero the first n floats of each layer (grid y = layers, grid-stride on x).
__global__ __launch_bounds__(kThreads) void k_zero_rows(float* __restrict__ p, size_t stride,
                                                       size_t n) {
  float* q = p + (size_t)blockIdx.y * stride;
  const size_t step = (size_t)gridDim.x * kThreads;
  for (size_t k = (size_t)blockIdx.x * kThreads + threadIdx.x; k < n; k += step) q[k] = 0.f;
}

inline unsigned blocks_for(int64_t n) { return (unsigned)((n + kThreads - 1) / kThreads); }

// Layers go on grid z (times the output split); launches are chunked over
// layers so that z stays within the 65536-block limit of y and z.
template <bool RED>
hipError_t dispatch_fused(int U, const float* y, float* z, float* S, const float* Hf,
                          const Shape& s, int t, int dst_len, hipStream_t st) {
  const dim3 block(kThreads);
#define LCSM_FUSED_CASE(UU)                                                                      \
  case UU: {                                                                                     \
    constexpr int SP = UU > 0 ? Split<UU>::value : 1;                                            \
    constexpr int MC = 65535 / SP;                                                               \
    for (int m0 = 0; m0 < s.M; m0 += MC) {                                                       \
      const int mc = s.M - m0 < MC ? s.M - m0 : MC;                                              \
      hipLaunchKernelGGL((k_step_fused<UU, RED>),                                                \
                         dim3(blocks_for(s.D), (unsigned)s.B, (unsigned)(mc * SP)), block, 0,    \
                         st, y, z, S, Hf, m0, s.L, s.SL, s.BD, s.D, t, dst_len);                \
    }                                                                                            \
    break;                                                                                       \
  }
  switch (U) {
    LCSM_FUSED_CASE(0)
    LCSM_FUSED_CASE(1)
    LCSM_FUSED_CASE(2)
    LCSM_FUSED_CASE(4)
    LCSM_FUSED_CASE(8)
    LCSM_FUSED_CASE(16)
    LCSM_FUSED_CASE(32)
    LCSM_FUSED_CASE(64)
    default:
      return hipErrorInvalidValue;
  }
#undef LCSM_FUSED_CASE
  return hipGetLastError();
}

}  // namespace

hipError_t launch_transpose_filters(const float* src, float* dst, const Shape& s, hipStream_t st) {
  const dim3 grid((s.D + 31) / 32, (s.L + 31) / 32, s.M);
  hipLaunchKernelGGL(k_transpose, grid, dim3(kThreads), 0, st, src, dst, s.D, s.L);
  return hipGetLastError();
}

hipError_t launch_step_fused(const float* y, float* z, float* S, const float* Hf, const Shape& s,
                             int t, int U, int dst_len, hipStream_t st) {
  return dispatch_fused<true>(U, y, z, S, Hf, s, t, dst_len, st);
}

hipError_t launch_chain_fused(const float* x, float* z, float* S, const float* Hf, float* prev,
                              const Shape& s, int t, int U, int dst_len, hipStream_t st) {
  const dim3 grid(blocks_for(s.D), (unsigned)s.B), block(kThreads);
#define LCSM_CHAIN_K(UU, KK)                                                                      \
  hipLaunchKernelGGL((k_chain_fused<UU, KK>), grid, block, 0, st, x, z, S, Hf, prev, s.M, s.L,   \
                     s.SL, s.BD, s.D, t, dst_len)
#define LCSM_CHAIN_CASE(UU)                                                                       \
  case UU: {                                                                                      \
    constexpr int KM = ChainChunk<UU>::value;                                                     \
    if (KM >= 8 && s.M >= 8) {                                                                    \
      LCSM_CHAIN_K(UU, (KM >= 8 ? 8 : 1));                                                        \
    } else if (KM >= 4 && s.M >= 4) {                                                             \
      LCSM_CHAIN_K(UU, (KM >= 4 ? 4 : 1));                                                        \
    } else if (KM >= 2 && s.M >= 2) {                                                             \
      LCSM_CHAIN_K(UU, (KM >= 2 ? 2 : 1));                                                        \
    } else {                                                                                      \
      LCSM_CHAIN_K(UU, 1);                                                                        \
    }                                                                                             \
    break;                                                                                        \
  }
  switch (U) {
    LCSM_CHAIN_CASE(0)
    LCSM_CHAIN_CASE(1)
    LCSM_CHAIN_CASE(2)
    LCSM_CHAIN_CASE(4)
    LCSM_CHAIN_CASE(8)
    LCSM_CHAIN_CASE(16)
    LCSM_CHAIN_CASE(32)
    default:
      return hipErrorInvalidValue;
  }
#undef LCSM_CHAIN_CASE
#undef LCSM_CHAIN_K
  return hipGetLastError();
}

hipError_t launch_chain_block(const float* x, size_t xst, int xring, int xs0, float* z,
                              size_t zst, int zring, int zs0, float* S, const float* Hf,
                              float* prev, const Shape& s, int t0, int t1, bool tile_last,
                              hipStream_t st) {
  if (s.M > kChainBlockMaxM || t1 <= t0 || (t0 & ~(kChainBlockW - 1)) != ((t1 - 1) & ~(kChainBlockW - 1)))
    return hipErrorInvalidValue;
  const int nw = 1 + (s.M + 1) / 2;
  const dim3 grid((unsigned)((s.BD + kChainBlockCols - 1) / kChainBlockCols)), block((unsigned)(64 * nw));
  if (s.M <= kChainBlockWave0StoreM)
    hipLaunchKernelGGL(k_chain_block<true>, grid, block, 0, st, x, xst, xring, xs0, z, zst, zring,
                       zs0, S, Hf, prev, s.M, s.L, s.SL, s.BD, s.D, t0, t1, tile_last ? 1 : 0);
  else
    hipLaunchKernelGGL(k_chain_block<false>, grid, block, 0, st, x, xst, xring, xs0, z, zst, zring,
                       zs0, S, Hf, prev, s.M, s.L, s.SL, s.BD, s.D, t0, t1, tile_last ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_red_layer(const float* y, float* z, float* S, const float* Hf, const Shape& s,
                            int layer, int t, hipStream_t st) {
  float* Sm = S + (size_t)layer * s.SL * s.BD;
  const float* Hm = Hf + (size_t)layer * s.L * s.D;
  hipLaunchKernelGGL(k_red_layer, dim3(blocks_for(s.BD)), dim3(kThreads), 0, st, y, z, Sm, Hm,
                     s.BD, s.D, t);
  return hipGetLastError();
}

hipError_t launch_direct_tile(float* S, const float* Hf, const Shape& s, int i, int U, int dst_len,
                              hipStream_t st) {
  if (dst_len <= 0) return hipSuccess;
  if (U <= kFusedMaxU) {
    // small tiles: whole tile per thread; position t = i-1 already holds y
    return dispatch_fused<false>(U, nullptr, nullptr, S, Hf, s, i - 1, dst_len, st);
  }
  const dim3 grid(blocks_for(s.BD), (dst_len + kDirectJ - 1) / kDirectJ, s.M);
  hipLaunchKernelGGL(k_direct_tile<kDirectJ>, grid, dim3(kThreads), 0, st, S, Hf, s.L, s.SL, s.BD,
                     s.D, i, U, dst_len);
  return hipGetLastError();
}

hipError_t launch_rows_in(const float* y, size_t y_stride, float* S, const Shape& s, int P,
                          hipStream_t st) {
  const size_t n = (size_t)P * s.M * s.BD;
  if (n == 0) return hipSuccess;
  size_t blocks = (n + kThreads - 1) / kThreads;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(k_rows_in, dim3((unsigned)blocks), dim3(kThreads), 0, st, y, y_stride, S, s.M,
                     s.SL, s.BD, P);
  return hipGetLastError();
}

hipError_t launch_rows_out_clear(float* S, const Shape& s, int row0, int P, float* z,
                                 size_t z_stride, hipStream_t st) {
  const size_t n = (size_t)P * s.M * s.BD;
  if (n == 0) return hipSuccess;
  size_t blocks = (n + kThreads - 1) / kThreads;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(k_rows_out_clear, dim3((unsigned)blocks), dim3(kThreads), 0, st, S, s.M, s.SL,
                     s.BD, row0, P, z, z_stride);
  return hipGetLastError();
}

hipError_t launch_zero_rows(float* p, int M, size_t stride, size_t n, hipStream_t st) {
  if (n == 0 || M <= 0) return hipSuccess;
  size_t bx = (n + kThreads - 1) / kThreads;
  const size_t cap = (8192 + (size_t)M - 1) / (size_t)M;  // about 8192 workgroups in all
  if (bx > cap) bx = cap;
  for (int m0 = 0; m0 < M; m0 += 65535) {
    const int mc = M - m0 < 65535 ? M - m0 : 65535;
    hipLaunchKernelGGL(k_zero_rows, dim3((unsigned)bx, (unsigned)mc), dim3(kThreads), 0, st,
                       p + (size_t)m0 * stride, stride, n);
  }
  return hipGetLastError();
}

hipError_t launch_zero(float* p, size_t n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  size_t blocks = (n + kThreads - 1) / kThreads;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(k_zero, dim3((unsigned)blocks), dim3(kThreads), 0, st, p, n);
  return hipGetLastError();
}

}  // namespace lcsm
