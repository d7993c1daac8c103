// Radix-16/8/4/2 Stockham FFT over columns held in LDS, for gfx950.
//
// A workgroup transforms WC complex columns of N points at once.  The LDS
// buffer is laid out [n][col] with a row stride of LDSW float2 (LDSW >= WC),
// so one row of the buffer is a contiguous run of the workgroup's columns and
// a wavefront touches consecutive 8-byte words.
//
// Pass structure (Stockham autosort, no bit reversal).  With p the product of
// the radices already applied (p = 1 before the first pass), a radix-R pass
// maps, for every j < N/R with k = j mod p,
//     u_q = x[j + q N/R] * w_{pR}^{q k}         (q < R)
//     x'[(j - k) R + k + s p] = sum_q u_q w_R^{q s}   (s < R)
// where w_n = exp(-2 pi i / n) for the forward and exp(+2 pi i / n) for the
// inverse transform (no 1/N factor).  After the last pass x' is the DFT in
// natural order.  The radices of an N-point transform are given by Plan<N>.
//
// Twiddles come from a table tw[n + m] = exp(-2 pi i m / n) for every power of
// two n (m < n), built on the host in double precision and rounded once.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

namespace lcsm {
namespace fft {

__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
  return make_float2(fmaf(a.x, b.x, -a.y * b.y), fmaf(a.x, b.y, a.y * b.x));
}
// a * conj(b)
__device__ __forceinline__ float2 cmulc(float2 a, float2 b) {
  return make_float2(fmaf(a.x, b.x, a.y * b.y), fmaf(a.y, b.x, -a.x * b.y));
}
__device__ __forceinline__ float2 conjf2(float2 a) { return make_float2(a.x, -a.y); }

// Twiddle w_n^e (forward sign) or its conjugate (inverse), 0 <= e < n, from
// the global table.
template <bool INV>
__device__ __forceinline__ float2 twiddle(const float2* __restrict__ tw, int n, int e) {
  const float2 w = tw[n + e];
  return INV ? conjf2(w) : w;
}

// Twiddle sources of the passes: the global table, or a copy of
// w_N^m (m < N) in LDS for an N-point transform (w_n^e = w_N^{e N/n}).
struct TwGlobal {
  const float2* __restrict__ t;
  template <bool INV, int NN>
  __device__ __forceinline__ float2 get(int e) const {
    return twiddle<INV>(t, NN, e);
  }
};

template <int N>
struct TwLds {
  const float2* t;
  template <bool INV, int NN>
  __device__ __forceinline__ float2 get(int e) const {
    const float2 w = t[e * (N / NN)];
    return INV ? conjf2(w) : w;
  }
};

// Half table: w_N^m for m < N/2 only, using w_N^{m + N/2} = -w_N^m (for an
// N-point transform whose data leaves no room for the full table).
template <int N>
struct TwLdsHalf {
  const float2* t;
  template <bool INV, int NN>
  __device__ __forceinline__ float2 get(int e) const {
    const int f = e * (N / NN);
    const float2 w = t[f & (N / 2 - 1)];
    const float s = (f & (N / 2)) ? -1.f : 1.f;
    return INV ? make_float2(s * w.x, -s * w.y) : make_float2(s * w.x, s * w.y);
  }
};

// A twiddle source with a member row<INV, NN, R>(k, w), filling w[q] =
// w_NN^{q k} for 0 < q < R in one call, gives the passes all twiddles of a
// butterfly at once (its own way of deriving them from fewer table reads);
// other sources are asked one twiddle at a time.
template <class TW, class = void>
struct HasRow : std::false_type {};
template <class TW>
struct HasRow<TW, std::void_t<decltype(TW::kRow)>> : std::true_type {};

template <bool INV, int NN, int R, class TW>
__device__ __forceinline__ void apply_twiddle_row(const TW& tw, int k, float2 (&v)[R]) {
  float2 w[R];
  tw.template row<INV, NN, R>(k, w);
#pragma unroll
  for (int q = 1; q < R; ++q) v[q] = cmul(v[q], w[q]);
}

// Copy w_N^m, m < NM, from the global table of the N-point twiddles into LDS
// (no synchronisation).
template <int N, int NT, int NM = N>
__device__ __forceinline__ void load_twiddles(float2* lds, const float2* __restrict__ tw) {
  for (int m = (int)threadIdx.x; m < NM; m += NT) lds[m] = tw[N + m];
}

// multiply by w_4 (forward -i, inverse +i)
template <bool INV>
__device__ __forceinline__ float2 rot90(float2 a) {
  return INV ? make_float2(-a.y, a.x) : make_float2(a.y, -a.x);
}
// multiply by w_8
template <bool INV>
__device__ __forceinline__ float2 rot45(float2 a) {
  constexpr float c = 0.70710678118654752440f;
  return INV ? make_float2(c * (a.x - a.y), c * (a.x + a.y)) : make_float2(c * (a.x + a.y), c * (a.y - a.x));
}
// multiply by w_8^3
template <bool INV>
__device__ __forceinline__ float2 rot135(float2 a) {
  constexpr float c = 0.70710678118654752440f;
  return INV ? make_float2(-c * (a.x + a.y), c * (a.x - a.y)) : make_float2(c * (a.y - a.x), -c * (a.x + a.y));
}

template <bool INV>
__device__ __forceinline__ void dft2(float2& a, float2& b) {
  const float2 t = a;
  a = cadd(t, b);
  b = csub(t, b);
}

template <bool INV>
__device__ __forceinline__ void dft4(float2& a0, float2& a1, float2& a2, float2& a3) {
  const float2 t0 = cadd(a0, a2), t1 = csub(a0, a2);
  const float2 t2 = cadd(a1, a3), t3 = rot90<INV>(csub(a1, a3));
  a0 = cadd(t0, t2);
  a2 = csub(t0, t2);
  a1 = cadd(t1, t3);
  a3 = csub(t1, t3);
}

// multiply by the constant w_16^e (e = 1 or 3; forward sign, conjugated for
// the inverse)
template <bool INV, int E>
__device__ __forceinline__ float2 rot16(float2 a) {
  constexpr float c1 = 0.92387953251128675613f;  // cos(pi/8)
  constexpr float s1 = 0.38268343236508977173f;  // sin(pi/8)
  constexpr float c = E == 1 ? c1 : s1;           // cos(E pi/8)
  constexpr float s = E == 1 ? s1 : c1;           // sin(E pi/8)
  // w = c - i s (forward), c + i s (inverse)
  return INV ? make_float2(c * a.x - s * a.y, c * a.y + s * a.x)
             : make_float2(c * a.x + s * a.y, c * a.y - s * a.x);
}

// In-place DFT of R points held in registers, natural order in and out.
// Radix 16 is four radix-4 DFTs over the stride-4 subsequences, the twiddles
// w_16^{n2 k1}, and four radix-4 DFTs across them.
template <int R, bool INV>
__device__ __forceinline__ void dft(float2* v) {
  if constexpr (R == 2) {
    dft2<INV>(v[0], v[1]);
  } else if constexpr (R == 4) {
    dft4<INV>(v[0], v[1], v[2], v[3]);
  } else if constexpr (R == 8) {
    float2 e0 = v[0], e1 = v[2], e2 = v[4], e3 = v[6];
    float2 o0 = v[1], o1 = v[3], o2 = v[5], o3 = v[7];
    dft4<INV>(e0, e1, e2, e3);
    dft4<INV>(o0, o1, o2, o3);
    o1 = rot45<INV>(o1);
    o2 = rot90<INV>(o2);
    o3 = rot135<INV>(o3);
    v[0] = cadd(e0, o0);
    v[4] = csub(e0, o0);
    v[1] = cadd(e1, o1);
    v[5] = csub(e1, o1);
    v[2] = cadd(e2, o2);
    v[6] = csub(e2, o2);
    v[3] = cadd(e3, o3);
    v[7] = csub(e3, o3);
  } else {
    static_assert(R == 16, "radix 2, 4, 8 or 16");
    // y[n2][k1] = sum_{n1} x[4 n1 + n2] w_4^{n1 k1}
    float2 y[4][4];
#pragma unroll
    for (int n2 = 0; n2 < 4; ++n2) {
      y[n2][0] = v[n2];
      y[n2][1] = v[4 + n2];
      y[n2][2] = v[8 + n2];
      y[n2][3] = v[12 + n2];
      dft4<INV>(y[n2][0], y[n2][1], y[n2][2], y[n2][3]);
    }
    // twiddles w_16^{n2 k1}: exponents 1 2 3 / 2 4 6 / 3 6 9
    y[1][1] = rot16<INV, 1>(y[1][1]);
    y[1][2] = rot45<INV>(y[1][2]);
    y[1][3] = rot16<INV, 3>(y[1][3]);
    y[2][1] = rot45<INV>(y[2][1]);
    y[2][2] = rot90<INV>(y[2][2]);
    y[2][3] = rot135<INV>(y[2][3]);
    y[3][1] = rot16<INV, 3>(y[3][1]);
    y[3][2] = rot135<INV>(y[3][2]);
    {
      const float2 w = rot16<INV, 1>(y[3][3]);  // w_16^9 = -w_16^1
      y[3][3] = make_float2(-w.x, -w.y);
    }
    // X[k1 + 4 k2] = sum_{n2} y[n2][k1] w_4^{n2 k2}
#pragma unroll
    for (int k1 = 0; k1 < 4; ++k1) {
      float2 a0 = y[0][k1], a1 = y[1][k1], a2 = y[2][k1], a3 = y[3][k1];
      dft4<INV>(a0, a1, a2, a3);
      v[k1] = a0;
      v[k1 + 4] = a1;
      v[k1 + 8] = a2;
      v[k1 + 12] = a3;
    }
  }
}

constexpr int ilog2(int n) { return n <= 1 ? 0 : 1 + ilog2(n / 2); }

// Radix plan of an N-point transform, as few passes as radices 16 and 8
// allow: radix-16 passes first (the very first may be radix 2 or 4 when
// neither fits exactly), then radix 8.  log2 N -> radices:
//   1..4: N;  5: 2 16;  6: 8 8;  7: 16 8;  8: 16 16;  9: 8 8 8;  10: 16 8 8;
//   11: 16 16 8;  12: 16 16 16;  13: 16 8 8 8;  and so on.
// With LCSM_RADIX8_ONLY defined: radix 8 throughout, radix 2 or 4 first.
template <int N>
struct Plan {
  static_assert(N >= 2 && (N & (N - 1)) == 0, "power of two");
  static constexpr int LOG = ilog2(N);
#ifdef LCSM_RADIX8_ONLY
  static constexpr int N16 = 0;
  static constexpr int N8 = LOG / 3;
  static constexpr int REM = LOG - 3 * N8;  // 0, 1 or 2
#else
  // number of radix-16 passes n16 and radix-8 passes n8 with 4 n16 + 3 n8 =
  // LOG - rem, minimising the pass count, rem in {0, 1, 2} only if needed
  static constexpr int pick(int what) {
    int best_np = 1 << 30, b16 = 0, b8 = 0, brem = 0;
    for (int rem = 0; rem <= 2; ++rem)
      for (int n16 = 0; 4 * n16 <= LOG - rem; ++n16) {
        const int left = LOG - rem - 4 * n16;
        if (left % 3) continue;
        const int n8 = left / 3;
        const int np = n16 + n8 + (rem ? 1 : 0);
        // fewer passes first, then no remainder pass, then fewer radix-16
        if (np < best_np || (np == best_np && rem < brem) ||
            (np == best_np && rem == brem && n16 < b16)) {
          best_np = np;
          b16 = n16;
          b8 = n8;
          brem = rem;
        }
      }
    return what == 0 ? b16 : (what == 1 ? b8 : brem);
  }
  static constexpr int N16 = LOG <= 4 ? 0 : pick(0);
  static constexpr int N8 = LOG <= 4 ? 0 : pick(1);
  static constexpr int REM = LOG <= 4 ? LOG : pick(2);  // LOG <= 4: one pass of radix N
#endif
  static constexpr int NP = N16 + N8 + (REM ? 1 : 0);
  static constexpr int radix(int ps) {
    return REM ? (ps == 0 ? (1 << REM) : (ps <= N16 ? 16 : 8)) : (ps < N16 ? 16 : 8);
  }
  // product of the radices of passes 0 .. ps-1
  static constexpr int p_before(int ps) {
    int p = 1;
    for (int k = 0; k < ps; ++k) p *= radix(k);
    return p;
  }
};

// LDS slot of element i: with SH > 0 one padding slot follows every 2^SH
// elements, which spreads the power-of-two strides of the butterfly outputs
// over the banks (a buffer of n elements then needs n + n / 2^SH slots).
template <int SH>
__device__ __forceinline__ int lds_slot(int i) {
  if constexpr (SH > 0) return i + (i >> SH);
  return i;
}

// Slot distance of an element distance that is a multiple of 2^SH (the
// padding below the element carries over), a constant where off is one: the
// passes take their unrolled accesses as immediate offsets from one slot.
template <int SH>
__device__ __forceinline__ int lds_step(int off) {
  if constexpr (SH > 0) return off + (off >> SH);
  return off;
}

// One radix-R pass (pass index PS of Plan<N>) in LDS, in place: every thread
// loads the inputs of all its butterflies, the workgroup synchronises, then
// every thread writes its outputs.  Callers synchronise before the first pass.
template <int N, int PS, int WC, int LDSW, int NT, bool INV, int SH = 0, class TW>
__device__ __forceinline__ void lds_pass(float2* buf, const TW& tw) {
  constexpr int R = Plan<N>::radix(PS);
  constexpr int P = Plan<N>::p_before(PS);
  constexpr int UNITS = N / R * WC;
  constexpr int UPT = (UNITS + NT - 1) / NT;
  float2 v[UPT][R];
#pragma unroll
  for (int a = 0; a < UPT; ++a) {
    const int u = (int)threadIdx.x + a * NT;
    if (UNITS % NT == 0 || u < UNITS) {
      const int j = u / WC, col = u % WC;
      if constexpr (SH == 0) {
#pragma unroll
        for (int q = 0; q < R; ++q) v[a][q] = buf[(j + q * (N / R)) * LDSW + col];
      } else {
        constexpr int ST = N / R * LDSW;
        const int b = lds_slot<SH>(j * LDSW + col);
#pragma unroll
        for (int q = 0; q < R; ++q) {
          if constexpr (ST % (1 << SH) == 0)
            v[a][q] = buf[b + lds_step<SH>(q * ST)];
          else
            v[a][q] = buf[lds_slot<SH>((j + q * (N / R)) * LDSW + col)];
        }
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int a = 0; a < UPT; ++a) {
    const int u = (int)threadIdx.x + a * NT;
    if (UNITS % NT == 0 || u < UNITS) {
      const int j = u / WC, col = u % WC;
      const int k = j & (P - 1);
      if constexpr (P > 1 && HasRow<TW>::value) {
        apply_twiddle_row<INV, P * R>(tw, k, v[a]);
      } else if constexpr (P > 1) {
#pragma unroll
        for (int q = 1; q < R; ++q) v[a][q] = cmul(v[a][q], tw.template get<INV, P * R>(q * k));
      }
      dft<R, INV>(v[a]);
      if constexpr (SH == 0) {
#pragma unroll
        for (int s = 0; s < R; ++s) buf[((j - k) * R + k + s * P) * LDSW + col] = v[a][s];
      } else {
        constexpr int PL = P * LDSW;
        const int b = lds_slot<SH>(((j - k) * R + k) * LDSW + col);
#pragma unroll
        for (int s = 0; s < R; ++s) {
          if constexpr (PL % (1 << SH) == 0)
            buf[b + lds_step<SH>(s * PL)] = v[a][s];
          else
            buf[lds_slot<SH>(((j - k) * R + k + s * P) * LDSW + col)] = v[a][s];
        }
      }
    }
  }
  __syncthreads();
}

template <int N, int PS, int PE, int WC, int LDSW, int NT, bool INV, int SH = 0, class TW>
__device__ __forceinline__ void lds_passes(float2* buf, const TW& tw) {
  if constexpr (PS < PE) {
    lds_pass<N, PS, WC, LDSW, NT, INV, SH>(buf, tw);
    lds_passes<N, PS + 1, PE, WC, LDSW, NT, INV, SH>(buf, tw);
  }
}

// First pass (index 0, p = 1, no twiddles) with inputs fetched by
// load(row, col) instead of from LDS; only rows < N*QIN/R are fetched (the
// rest are zero: QIN = R/2 for a zero-padded upper half, R for full input).
// Writes its outputs to LDS and synchronises.
template <int N, int WC, int LDSW, int NT, bool INV, bool HALF, int SH = 0, class Load>
__device__ __forceinline__ void first_pass_global(float2* buf, const Load& load) {
  constexpr int R = Plan<N>::radix(0);
  constexpr int QIN = HALF ? R / 2 : R;
  constexpr int UNITS = N / R * WC;
  constexpr int UPT = (UNITS + NT - 1) / NT;
  float2 v[UPT][R];
#pragma unroll
  for (int a = 0; a < UPT; ++a) {
    const int u = (int)threadIdx.x + a * NT;
    if (UNITS % NT == 0 || u < UNITS) {
      const int j = u / WC, col = u % WC;
#pragma unroll
      for (int q = 0; q < R; ++q) v[a][q] = (q < QIN) ? load(j + q * (N / R), col) : make_float2(0.f, 0.f);
    }
  }
#pragma unroll
  for (int a = 0; a < UPT; ++a) {
    const int u = (int)threadIdx.x + a * NT;
    if (UNITS % NT == 0 || u < UNITS) {
      const int j = u / WC, col = u % WC;
      dft<R, INV>(v[a]);
      if constexpr (SH == 0) {
#pragma unroll
        for (int s = 0; s < R; ++s) buf[(j * R + s) * LDSW + col] = v[a][s];
      } else {
        // one column only: j R is a multiple of R, so for s < R the slot of
        // j R + s is that of j R plus s plus the padding within s
        static_assert(LDSW == 1, "padded LDS holds one column");
        const int b = lds_slot<SH>(j * R);
#pragma unroll
        for (int s = 0; s < R; ++s) {
          if constexpr (R <= (1 << SH))
            buf[b + s] = v[a][s];
          else
            buf[b + s + (s >> SH)] = v[a][s];
        }
      }
    }
  }
  __syncthreads();
}

// Last pass (index NP-1, p = N/R) reading LDS and handing the outputs of
// rows >= N/2 (HALF) or of all rows to store(row, col, value) instead of
// writing LDS.  No synchronisation at the end (LDS is only read).
template <int N, int WC, int LDSW, int NT, bool INV, bool HALF, int SH = 0, class TW,
          class Store>
__device__ __forceinline__ void last_pass_global(const float2* buf, const TW& tw,
                                                 const Store& store) {
  constexpr int PS = Plan<N>::NP - 1;
  constexpr int R = Plan<N>::radix(PS);
  constexpr int P = Plan<N>::p_before(PS);
  static_assert(P * R == N, "last pass");
  constexpr int UNITS = N / R * WC;
  constexpr int UPT = (UNITS + NT - 1) / NT;
  constexpr int S0 = HALF ? R / 2 : 0;
#pragma unroll
  for (int a = 0; a < UPT; ++a) {
    const int u = (int)threadIdx.x + a * NT;
    if (UNITS % NT == 0 || u < UNITS) {
      const int j = u / WC, col = u % WC;  // j < P, so k = j
      float2 v[R];
      if constexpr (SH == 0) {
#pragma unroll
        for (int q = 0; q < R; ++q) v[q] = buf[(j + q * (N / R)) * LDSW + col];
      } else {
        constexpr int ST = N / R * LDSW;
        const int b = lds_slot<SH>(j * LDSW + col);
#pragma unroll
        for (int q = 0; q < R; ++q) {
          if constexpr (ST % (1 << SH) == 0)
            v[q] = buf[b + lds_step<SH>(q * ST)];
          else
            v[q] = buf[lds_slot<SH>((j + q * (N / R)) * LDSW + col)];
        }
      }
      if constexpr (P > 1 && HasRow<TW>::value) {
        apply_twiddle_row<INV, N>(tw, j, v);
      } else if constexpr (P > 1) {
#pragma unroll
        for (int q = 1; q < R; ++q) v[q] = cmul(v[q], tw.template get<INV, N>(q * j));
      }
      dft<R, INV>(v);
#pragma unroll
      for (int s = S0; s < R; ++s) store(j + s * P, col, v[s]);
    }
  }
}

// Forward transform whose input is fetched by load(): first pass from
// global, the rest in LDS.  Result in LDS, natural order.
template <int N, int WC, int LDSW, int NT, bool HALF, int SH = 0, class TW, class Load>
__device__ __forceinline__ void forward_from_global(float2* buf, const TW& tw, const Load& load) {
  first_pass_global<N, WC, LDSW, NT, false, HALF, SH>(buf, load);
  lds_passes<N, 1, Plan<N>::NP, WC, LDSW, NT, false, SH>(buf, tw);
}

// Inverse transform of the LDS contents whose outputs go to store() (rows >=
// N/2 only when HALF).  The caller synchronises before.
template <int N, int WC, int LDSW, int NT, bool HALF, int SH = 0, class TW, class Store>
__device__ __forceinline__ void inverse_to_global(float2* buf, const TW& tw, const Store& store) {
  lds_passes<N, 0, Plan<N>::NP - 1, WC, LDSW, NT, true, SH>(buf, tw);
  last_pass_global<N, WC, LDSW, NT, true, HALF, SH>(buf, tw, store);
}

// Hardware dispatches workgroup b to XCD b mod 8.  Remap so that XCD x runs a
// contiguous range of logical workgroup ids (neighbours then share that
// XCD's L2).  A bijection on [0, nb).
__device__ __forceinline__ int xcd_logical(int b, int nb) {
  const int per = nb / 8;
  if (b >= per * 8) return b;
  return (b % 8) * per + b / 8;
}

}  // namespace fft
}  // namespace lcsm
