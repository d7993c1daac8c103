// FFT gray tiles and filter spectra of the relaxed online convolution, for
// gfx950.
//
// A gray tile of side U (Eq. taus) adds, for j < U,
//     z[i+j] += sum_{k<U} y[i-U+k] h[U+j-k]
// Lemma 1 with the cyclic shortcut of App. B: right-pad the U inputs with U
// zeros, multiply the N = 2U point DFT with the DFT of the filter prefix
// h[0, N), and invert; outputs U..N-1 of the cyclic convolution are the
// wanted ones (the wrap-around only reaches outputs < U-1).  The filter DFTs
// are computed once per tile size at initialisation (the cached kernel DFTs
// of Sec. 5 / App. B) and stored pre-scaled by 1/N.
//
// Two real columns are carried in one complex signal: real part column c,
// imaginary part column c+1 (one float2 load per row).  If Z is the DFT of
// the pair and Ha, Hb the filter spectra of the two columns, the spectrum of
// (conv(a, ha) + i conv(b, hb)) is
//     P[k] = Z[k] S[k] + conj(Z[N-k]) D[k],   S = (Ha+Hb)/2,  D = (Ha-Hb)/2,
// which needs the bins k and N-k together.
//
// Data layout: state S[m][t][c] (c = b*D + d, row stride B*D), filters
// Hf[m][k][d], spectra of tile size U: H[m][k][d] complex, k = 0..U (the
// other bins follow from conjugate symmetry).
//
// Single pass (N <= LDS limit): one workgroup owns WC complex columns and all
// N points in LDS; it reads the U input rows once and adds into the U output
// rows once.
//
// Multi pass (larger N), a four-step split N = N1 N2 with time index
// n = n1 + N1 n2 and frequency index k = N2 k1 + k2:
//   pass R  : for each n1 an N2-point FFT over the rows n1 + N1 n2 of the
//             block (only n2 < N2/2 are non-zero), times w_N^{n1 k2} -> C
//   pass M  : for each k2 an N1-point DFT over n1 (giving X[N2 k1 + k2]),
//             the spectral product (partner bin N-k lies in column N2-k2),
//             the inverse N1-point DFT and the conjugate twiddle, in place
//   pass R' : for each n1 the inverse N2-point FFT of C; outputs n2 >= N2/2
//             are the time indices U..N-1, added into the state.
// C lives in a scratch buffer; columns are processed in chunks.
#include <type_traits>

#include "lcsm_fft_core.h"
#include "lcsm_internal.h"

namespace lcsm {
namespace {

using fft::cadd;
using fft::cmul;
using fft::cmulc;
using fft::conjf2;
using fft::csub;

// Per-size launch shape of the LDS transforms: WC complex columns per
// workgroup, NT threads.  WC * 8 bytes is the contiguous run read and written
// per state row.  For 2U >= 1024 the tile kernels are bound by these strided
// row accesses far more than by the transforms (without any LDS pass they
// run barely faster), and narrow runs are expensive, so panels are as wide as
// LDS allows: 64-byte runs up to 2U = 2048, 32 at 4096, 16 at 8192.  TWL:
// the twiddle table w_N^m fits in LDS beside the data; TWH: only its first
// half does (the rest follows from w_N^{m+N/2} = -w_N^m).
template <int N>
struct Cfg {
  static constexpr int WC = N <= 256 ? 4 : (N <= 2048 ? 8 : (N <= 4096 ? 4 : 2));
  static constexpr int NT = N <= 128 ? 64 : (N <= 256 ? 128 : (N <= 512 ? 256 : (N <= 1024 ? 512 : (N <= 2048 ? 1024 : (N <= 4096 ? 512 : 1024)))));
  static constexpr bool TWL = (size_t)N * 8 * (WC + 1) <= 163840;
  static constexpr bool TWH = !TWL && (size_t)N * 8 * WC + (size_t)N * 4 <= 163840;
  static constexpr int TWN = TWL ? N : (TWH ? N / 2 : 1);  // LDS twiddle entries
};

// Twiddle source of an N-point transform: LDS copy (whole or half) when it
// fits, else the global table.  The LDS copy is written here and read after
// the caller's next __syncthreads.
template <int N>
using TwOf = typename std::conditional<
    Cfg<N>::TWL, fft::TwLds<N>,
    typename std::conditional<Cfg<N>::TWH, fft::TwLdsHalf<N>, fft::TwGlobal>::type>::type;

template <int N>
__device__ __forceinline__ TwOf<N> make_tw(float2* lds, const float2* __restrict__ tw) {
  if constexpr (Cfg<N>::TWL) {
    fft::load_twiddles<N, Cfg<N>::NT>(lds, tw);
    return fft::TwLds<N>{lds};
  } else if constexpr (Cfg<N>::TWH) {
    fft::load_twiddles<N, Cfg<N>::NT, N / 2>(lds, tw);
    return fft::TwLdsHalf<N>{lds};
  } else {
    return fft::TwGlobal{tw};
  }
}

// Pair load / accumulate of real columns c, c+1 of a row.
__device__ __forceinline__ float2 load_pair(const float* __restrict__ row, int c, int ncols, bool vec) {
  if (c >= ncols) return make_float2(0.f, 0.f);
  if (vec) return *reinterpret_cast<const float2*>(row + c);
  return make_float2(row[c], c + 1 < ncols ? row[c + 1] : 0.f);
}

__device__ __forceinline__ void add_pair(float* row, int c, int ncols, bool vec, float2 v) {
  if (c >= ncols) return;
  if (vec) {
    float2* p = reinterpret_cast<float2*>(row + c);
    float2 o = *p;
    o.x += v.x;
    o.y += v.y;
    *p = o;
  } else {
    row[c] += v.x;
    if (c + 1 < ncols) row[c + 1] += v.y;
  }
}

// Spectral product of the column pair (a, b) at bin k given Z[k] and
// Z[N-k]: returns P[k] (see the file header).
__device__ __forceinline__ float2 pair_product(float2 zk, float2 znk, float2 ha, float2 hb) {
  const float2 s = make_float2(0.5f * (ha.x + hb.x), 0.5f * (ha.y + hb.y));
  const float2 d = make_float2(0.5f * (ha.x - hb.x), 0.5f * (ha.y - hb.y));
  return cadd(cmul(zk, s), cmul(conjf2(znk), d));
}

// Panel of the r-th workgroup of a layer (panels of WC complex columns).  The
// LG panels that share 128-byte lines of a state row are consecutive
// (adjacent workgroups run together on one XCD, so each line is fetched and
// written back whole), and these line groups cycle through the batch rows of
// the same channels (which share the filter spectrum in L2).  hgroup = panels
// per batch row when D is a multiple of the panel width, else 0.  A bijection
// on [0, panels per layer).
template <int WC>
__device__ __forceinline__ int panel_of(int r, int B, int hgroup) {
  constexpr int LG = WC >= 16 ? 1 : 16 / WC;
  if (hgroup > 0 && hgroup % LG == 0) {
    const int g = r / LG;
    return (g % B) * hgroup + (g / B) * LG + (r - g * LG);
  }
  if (hgroup > 0) return (r % B) * hgroup + r / B;
  return r;
}

// ----------------------------------------------------------- single pass

// Every global load of a stage is issued before that stage needs it: the
// spectrum bins of the spectral product right after the first forward pass
// (in flight during the other forward passes), and the destination rows of
// the last inverse pass before the inverse passes start.  Without this the
// per-unit loads in loops that also store would each cost a full round trip.
//
// RED: the red cell of position t = i-1 is fused in.  Each workgroup first
// finalises z_t = fmaf(h_0, y_t, acc_t) for its own columns and stores y_t
// into state row t; its first forward pass takes block row U-1 (= row t)
// from the caller's y_t instead of the state, so no thread reads a value
// another thread of the launch has just written.
//
// FAST: every panel is whole and lies inside one batch row (D a multiple of
// 2 WC) and the destination is not clipped (dst_len = U).  Then no access
// needs a bounds check, the channel of a panel column is d0 + 2 col with d0
// computed once, and the two filter spectra of a column pair are adjacent
// (one 16-byte load).
// STORE (not with RED): the outputs are stored over the input rows [i-U,
// i-U+dst_len) instead of added into rows [i, i+dst_len).  The workgroup has
// read all inputs of its columns (the first pass, before the barriers of the
// LDS passes) before it stores, and no other workgroup touches its columns.
template <int N, bool RED, bool FAST, bool STORE = false, int WCX = Cfg<N>::WC>
__global__ __launch_bounds__(Cfg<N>::NT) void k_fft_tile(float* __restrict__ S,
                                                         const float2* __restrict__ H,
                                                         const float2* __restrict__ tw,
                                                         const float* __restrict__ Hf,
                                                         const float* __restrict__ yt,
                                                         float* __restrict__ zt, int L, int SL,
                                                         int BD, int D, int B, int i, int dst_len,
                                                         int ppl, int hgroup) {
  static_assert(!(RED && STORE), "the in-place store has no red cell");
  constexpr int WC = WCX, NT = Cfg<N>::NT, U = N / 2;
  using P = fft::Plan<N>;
  __shared__ float2 buf[N * WC];
  __shared__ float2 twl[Cfg<N>::TWN];
  const auto twz = make_tw<N>(twl, tw);
  const int q = fft::xcd_logical((int)blockIdx.x, (int)gridDim.x);
  const int m = q / ppl;
  const int c0 = panel_of<WC>(q - m * ppl, B, hgroup) * 2 * WC;
  const int d0 = FAST ? c0 % D : 0;
  const bool vec = FAST || (BD & 1) == 0;
  float* Sm = S + (size_t)m * SL * BD;
  const float* ysrc = Sm + (size_t)(i - U) * BD;
  const float* ym = RED ? yt + (size_t)m * BD : nullptr;
  const int dlen = FAST ? U : dst_len;

  if constexpr (RED) {
    const int t = i - 1;
    for (int k = (int)threadIdx.x; k < 2 * WC; k += NT) {
      const int c = c0 + k;
      if (FAST || c < BD) {
        const float y = ym[c];
        float* slot = Sm + (size_t)t * BD + c;
        zt[(size_t)m * BD + c] = fmaf(Hf[(size_t)m * L * D + (FAST ? d0 + k : c % D)], y, *slot);
        *slot = y;
      }
    }
  }

  // forward: first pass straight from the input rows
  fft::first_pass_global<N, WC, WC, NT, false, true>(buf, [&](int row, int col) {
    const float* src = (RED && row == U - 1) ? ym : ysrc + (size_t)row * BD;
    if constexpr (FAST) return *reinterpret_cast<const float2*>(src + c0 + 2 * col);
    return load_pair(src, c0 + 2 * col, BD, vec);
  });

  // spectrum bins kk = 0..U of this thread's product units, loaded before
  // the remaining forward passes when the registers allow it (2U <= 4096)
  constexpr int PUN = (U + 1) * WC;
  constexpr int PU = (PUN + NT - 1) / NT;
  constexpr bool PREH = N <= 4096;
  constexpr int PH = PREH ? PU : 1;
  const float2* Hm = H + (size_t)m * (U + 1) * D;
  // spectra of the column pair (c, c+1) at bin kk
  auto load_h = [&](int kk, int col, float2& xa, float2& xb) {
    if constexpr (FAST) {
      const float4 v = *reinterpret_cast<const float4*>(Hm + (size_t)kk * D + d0 + 2 * col);
      xa = make_float2(v.x, v.y);
      xb = make_float2(v.z, v.w);
    } else {
      const int c = c0 + 2 * col;
      xa = xb = make_float2(0.f, 0.f);
      if (c < BD) {
        const int da = c % D;
        const int db = (c + 1 < BD) ? (c + 1) % D : da;
        xa = Hm[(size_t)kk * D + da];
        xb = Hm[(size_t)kk * D + db];
      }
    }
  };
  float2 ha[PH], hb[PH];
  if constexpr (PREH) {
#pragma unroll
    for (int a = 0; a < PU; ++a) {
      const int u = (int)threadIdx.x + a * NT;
      const int kk = u / WC, col = u - kk * WC;
      ha[a] = hb[a] = make_float2(0.f, 0.f);
      if (PUN % NT == 0 || u < PUN) load_h(kk, col, ha[a], hb[a]);
    }
  }
  fft::lds_passes<N, 1, P::NP, WC, WC, NT, false>(buf, twz);

#pragma unroll
  for (int a = 0; a < PU; ++a) {
    const int u = (int)threadIdx.x + a * NT;
    if (PUN % NT == 0 || u < PUN) {
      const int kk = u / WC, col = u - kk * WC;
      float2 xa, xb;
      if constexpr (PREH) {
        xa = ha[a];
        xb = hb[a];
      } else {
        load_h(kk, col, xa, xb);
      }
      const int nk = (N - kk) & (N - 1);
      const float2 zk = buf[kk * WC + col], znk = buf[nk * WC + col];
      buf[kk * WC + col] = pair_product(zk, znk, xa, xb);
      if (nk != kk) buf[nk * WC + col] = pair_product(znk, zk, conjf2(xa), conjf2(xb));
    }
  }

  // destination rows of the last inverse pass (radix RL, p = N/RL): unit j
  // writes rows j + s N/RL for s >= RL/2, i.e. outputs oi = j + (s - RL/2) N/RL
  constexpr int RL = P::radix(P::NP - 1);
  constexpr int PL = N / RL;
  constexpr int LUN = PL * WC;
  constexpr int LU = (LUN + NT - 1) / NT;
  float* zdst = Sm + (size_t)(STORE ? i - U : i) * BD;
  constexpr bool PREZ = N <= 4096 && !STORE;  // registers allow the prefetch
  auto load_z = [&](int oi, int c) -> float2 {
    if constexpr (FAST) return *reinterpret_cast<const float2*>(zdst + (size_t)oi * BD + c);
    return load_pair(zdst + (size_t)oi * BD, c, BD, vec);
  };
  float2 zo[PREZ ? LU : 1][RL / 2];
  if constexpr (PREZ) {
#pragma unroll
    for (int a = 0; a < LU; ++a) {
      const int u = (int)threadIdx.x + a * NT;
      const int j = u / WC, col = u - j * WC;
#pragma unroll
      for (int s = 0; s < RL / 2; ++s) {
        const int oi = j + s * PL;
        zo[a][s] = ((LUN % NT == 0 || u < LUN) && (FAST || oi < dlen)) ? load_z(oi, c0 + 2 * col)
                                                                       : make_float2(0.f, 0.f);
      }
    }
  }
  __syncthreads();
  fft::lds_passes<N, 0, P::NP - 1, WC, WC, NT, true>(buf, twz);

#pragma unroll
  for (int a = 0; a < LU; ++a) {
    const int u = (int)threadIdx.x + a * NT;
    if (LUN % NT == 0 || u < LUN) {
      const int j = u / WC, col = u - j * WC;  // j < PL, so k = j
      float2 v[RL];
#pragma unroll
      for (int t = 0; t < RL; ++t) v[t] = buf[(j + t * PL) * WC + col];
      if constexpr (PL > 1) {
#pragma unroll
        for (int t = 1; t < RL; ++t) v[t] = cmul(v[t], twz.template get<true, N>(t * j));
      }
      fft::dft<RL, true>(v);
      const int c = c0 + 2 * col;
#pragma unroll
      for (int s = 0; s < RL / 2; ++s) {
        const int oi = j + s * PL;
        if (FAST || (oi < dlen && c < BD)) {
          float2 o = v[RL / 2 + s];
          if constexpr (!STORE) {
            const float2 zz = PREZ ? zo[PREZ ? a : 0][s] : load_z(oi, c);
            o = make_float2(zz.x + o.x, zz.y + o.y);
          }
          float* row = zdst + (size_t)oi * BD;
          if (vec) {
            *reinterpret_cast<float2*>(row + c) = o;
          } else {
            row[c] = o.x;
            if (c + 1 < BD) row[c + 1] = o.y;
          }
        }
      }
    }
  }
}

// Filter spectra of tile size U = N/2 for all layers: H[m][k][d] =
// DFT_N(g[m][0..N), d)[k] / N for k <= N/2, where g is the filter delayed by
// shift rows (g[r] = h[r - shift], zero before; taps at lags >= L are zero).
// shift = 0 for the tile spectra; shift = U for the prompt's own outputs.
template <int N>
__global__ __launch_bounds__(Cfg<N>::NT) void k_fft_spectra(const float* __restrict__ Hf,
                                                            float2* __restrict__ Hout,
                                                            const float2* __restrict__ tw, int L,
                                                            int D, int ppl, int shift, int colmaj) {
  constexpr int WC = Cfg<N>::WC, NT = Cfg<N>::NT, U = N / 2;
  __shared__ float2 buf[N * WC];
  __shared__ float2 twl[Cfg<N>::TWN];
  const auto twz = make_tw<N>(twl, tw);
  const int m = (int)blockIdx.x / ppl;
  const int c0 = ((int)blockIdx.x - m * ppl) * 2 * WC;
  const bool vec = (D & 1) == 0;
  const float* src = Hf + (size_t)m * L * D;
  fft::forward_from_global<N, WC, WC, NT, false>(buf, twz, [&](int row, int col) {
    const int hr = row - shift;  // the filter delayed by shift rows
    return (hr >= 0 && hr < L) ? load_pair(src + (size_t)hr * D, c0 + 2 * col, D, vec)
                               : make_float2(0.f, 0.f);
  });
  constexpr float inv_n = 1.0f / (float)N;
  float2* Hm = Hout + (size_t)m * (U + 1) * D;
  // [k][d] within the layer, or [d][k] (colmaj) for the column tiles
  const size_t sk = colmaj ? 1 : (size_t)D, sd = colmaj ? (size_t)(U + 1) : 1;
  for (int u = (int)threadIdx.x; u < (U + 1) * WC; u += NT) {
    const int kk = u / WC, col = u - kk * WC;
    const int c = c0 + 2 * col;
    if (c >= D) continue;
    const float2 a = buf[kk * WC + col], b = buf[((N - kk) & (N - 1)) * WC + col];
    Hm[kk * sk + c * sd] = make_float2(0.5f * inv_n * (a.x + b.x), 0.5f * inv_n * (a.y - b.y));
    if (c + 1 < D)
      Hm[kk * sk + (c + 1) * sd] =
          make_float2(0.5f * inv_n * (a.y + b.y), -0.5f * inv_n * (a.x - b.x));
  }
}

// ------------------------------------------------------------ multi pass

// Geometry of a multi-pass launch over one chunk of complex columns.
// Complex column g (global over layers) is layer g / ncc, real columns
// 2 (g % ncc) and 2 (g % ncc) + 1 of that layer.  Scratch element (row r,
// chunk column x) sits at r * cstride + x.
struct Chunk {
  int g0;       // first complex column of the chunk
  int nvalid;   // complex columns in the chunk
  int cstride;  // scratch row stride (complex columns, >= nvalid)
  int ncc;      // complex columns per layer = ceil(ncols / 2)
  int ncols;    // real columns per layer (B*D for the state, D for filters)
  int N1, N2;
};

// Pass R: N2-point FFT over rows row0 + n1 + N1 n2 of every layer's matrix
// (src + m*lstride, row stride ncols), rows < 0 or >= rows_valid read as zero; HALF:
// only n2 < N2/2 are read.  Output C[n1*N2 + k2][x] = FFT[k2] * w_N^{n1 k2}.
template <int N2, bool HALF>
__global__ __launch_bounds__(Cfg<N2>::NT) void k_fft_rows_fwd(const float* __restrict__ src,
                                                              size_t lstride, int row0,
                                                              int rows_valid, Chunk ch,
                                                              float2* __restrict__ C,
                                                              const float2* __restrict__ tw) {
  constexpr int WC = Cfg<N2>::WC, NT = Cfg<N2>::NT;
  __shared__ float2 buf[N2 * WC];
  __shared__ float2 twl[Cfg<N2>::TWN];
  const auto twz = make_tw<N2>(twl, tw);
  const int npan = (ch.nvalid + WC - 1) / WC;
  const int q = fft::xcd_logical((int)blockIdx.x, (int)gridDim.x);
  const int n1 = q / npan;
  const int x0 = (q - n1 * npan) * WC;
  const bool vec = (ch.ncols & 1) == 0;
  fft::forward_from_global<N2, WC, WC, NT, HALF>(buf, twz, [&](int n2, int col) {
    const int x = x0 + col;
    const int row = row0 + n1 + ch.N1 * n2;
    if (x >= ch.nvalid || row < 0 || row >= rows_valid) return make_float2(0.f, 0.f);
    const int g = ch.g0 + x;
    const int m = g / ch.ncc;
    const int c = 2 * (g - m * ch.ncc);
    return load_pair(src + m * lstride + (size_t)row * ch.ncols, c, ch.ncols, vec);
  });
  const int N = ch.N1 * N2;
  for (int u = (int)threadIdx.x; u < N2 * WC; u += NT) {
    const int k2 = u / WC, col = u - k2 * WC;
    const int x = x0 + col;
    if (x >= ch.nvalid) continue;
    C[(size_t)(n1 * N2 + k2) * ch.cstride + x] = cmul(buf[k2 * WC + col], fft::twiddle<false>(tw, N, n1 * k2));
  }
}

constexpr int kMidG = 8;   // frequency columns k2 per pass-M workgroup
constexpr int kMidWC = 8;  // complex columns per pass-M workgroup
constexpr int kMidNT = 256;

// Pass M of the filter spectra: C holds, per filter column pair, the
// pass-R pieces of DFT_N(h[0, N)).  Workgroup (kg, panel) owns the frequency
// columns k2 = kg*G + s (s < G) of complex columns x0 .. x0+WCM-1 and reads
// their partner columns N2 - k2 as well (LDS slot s holds k2, slot G + s its
// partner).  X = DFT_N1(C); the two real filters of each pair are separated
// and their 1/N-scaled spectra at bins k <= N/2 are written to Hout[m][k][d].
template <int N1>
__global__ __launch_bounds__(kMidNT) void k_fft_mid_spectra(const float2* __restrict__ C,
                                                            float2* __restrict__ Hout, int D,
                                                            Chunk ch,
                                                            const float2* __restrict__ tw,
                                                            int colmaj) {
  constexpr int G = kMidG, WCM = kMidWC, NT = kMidNT;
  constexpr int W = 2 * G * WCM;  // LDS row stride
  __shared__ float2 buf[N1 * W];
  __shared__ float2 twl[N1];
  const fft::TwLds<N1> twz{twl};
  fft::load_twiddles<N1, NT>(twl, tw);
  const int N2 = ch.N2, N = N1 * N2, U = N / 2;
  const int npan = (ch.nvalid + WCM - 1) / WCM;
  const int q = fft::xcd_logical((int)blockIdx.x, (int)gridDim.x);
  const int kg = q / npan;
  const int x0 = (q - kg * npan) * WCM;
  const int kA = kg * G;

  for (int u = (int)threadIdx.x; u < N1 * W; u += NT) {
    const int n1 = u / W, slot = (u - n1 * W) / WCM, cc = u % WCM;
    const int s = slot % G;
    const int k2 = slot < G ? kA + s : (N2 - kA - s) & (N2 - 1);
    const int x = x0 + cc;
    buf[u] = x < ch.nvalid ? C[(size_t)(n1 * N2 + k2) * ch.cstride + x] : make_float2(0.f, 0.f);
  }
  __syncthreads();
  fft::lds_passes<N1, 0, fft::Plan<N1>::NP, W, W, NT, false>(buf, twz);

  const float inv_n = 1.0f / (float)N;
  for (int u = (int)threadIdx.x; u < N1 * G * WCM; u += NT) {
    const int k1 = u / (G * WCM), sc = u - k1 * (G * WCM);
    const int s = sc / WCM, cc = sc - s * WCM;
    const int x = x0 + cc;
    if (x >= ch.nvalid) continue;
    const int k2 = kA + s;
    const int k = N2 * k1 + k2;
    if (k > U) continue;
    const int pk1 = k2 == 0 ? (N1 - k1) & (N1 - 1) : N1 - 1 - k1;
    const float2 xk = buf[k1 * W + s * WCM + cc];
    const float2 xp = buf[pk1 * W + (G + s) * WCM + cc];
    const int g = ch.g0 + x;
    const int m = g / ch.ncc;
    const int c = 2 * (g - m * ch.ncc);
    float2* Hm = Hout + (size_t)m * (U + 1) * D;
    const size_t sk = colmaj ? 1 : (size_t)D, sd = colmaj ? (size_t)(U + 1) : 1;
    Hm[k * sk + c * sd] = make_float2(0.5f * inv_n * (xk.x + xp.x), 0.5f * inv_n * (xk.y - xp.y));
    if (c + 1 < D)
      Hm[k * sk + (c + 1) * sd] =
          make_float2(0.5f * inv_n * (xk.y + xp.y), -0.5f * inv_n * (xk.x - xp.x));
  }
}

// Pass M of a tile, in place in C.  Workgroup group 0 owns the two
// self-paired frequency columns k2 = 0 and N2/2; group g >= 1 owns
// k2 = 1 + (g-1) G + s (s < G, k2 < N2/2) and their partners N2 - k2, so each
// column and each spectrum bin is read once.  LDS slot s < G holds k2_s,
// slot G + s its partner; the partner of bin (k1, slot s) is (N1-1-k1, slot
// G+s).  Per column: X = DFT_N1(C), spectral product, E = IDFT_N1(P) times
// conj(w_N^{n1 k2}), written back over C.
__device__ __forceinline__ int mid_slot_k2(int gi, int slot, int N2) {
  constexpr int G = kMidG;
  if (gi == 0) return slot == 0 ? 0 : (slot == 1 ? N2 / 2 : -1);
  const int s = slot < G ? slot : slot - G;
  const int k = 1 + (gi - 1) * G + s;
  if (k >= N2 / 2) return -1;
  return slot < G ? k : N2 - k;
}

template <int N1>
__global__ __launch_bounds__(kMidNT) void k_fft_mid_tile(float2* __restrict__ C,
                                                         const float2* __restrict__ H, int D,
                                                         Chunk ch, const float2* __restrict__ tw) {
  constexpr int G = kMidG, WCM = kMidWC, NT = kMidNT;
  constexpr int W = 2 * G * WCM;  // LDS row stride
  __shared__ float2 buf[N1 * W];
  __shared__ float2 twl[N1];
  const fft::TwLds<N1> twz{twl};
  fft::load_twiddles<N1, NT>(twl, tw);
  const int N2 = ch.N2, N = N1 * N2, U = N / 2;
  const int npan = (ch.nvalid + WCM - 1) / WCM;
  const int q = fft::xcd_logical((int)blockIdx.x, (int)gridDim.x);
  const int gi = q / npan;
  const int x0 = (q - gi * npan) * WCM;

  for (int u = (int)threadIdx.x; u < N1 * W; u += NT) {
    const int n1 = u / W, slot = (u - n1 * W) / WCM, cc = u % WCM;
    const int k2 = mid_slot_k2(gi, slot, N2);
    const int x = x0 + cc;
    buf[u] = (k2 >= 0 && x < ch.nvalid) ? C[(size_t)(n1 * N2 + k2) * ch.cstride + x] : make_float2(0.f, 0.f);
  }
  __syncthreads();
  fft::lds_passes<N1, 0, fft::Plan<N1>::NP, W, W, NT, false>(buf, twz);

  // spectral product over disjoint bin pairs (k, N-k)
  const int BD = ch.ncols;
  auto spectrum = [&](int m, int c, int k, float2& ha, float2& hb) {
    const int da = c % D;
    const int db = (c + 1 < BD) ? (c + 1) % D : da;
    const float2* Hm = H + (size_t)m * (U + 1) * D;
    const int kb = k <= U ? k : N - k;
    ha = Hm[(size_t)kb * D + da];
    hb = Hm[(size_t)kb * D + db];
    if (k > U) {
      ha = conjf2(ha);
      hb = conjf2(hb);
    }
  };
  auto pair = [&](int ia, int ib, int k, int m, int c) {
    float2 ha, hb;
    spectrum(m, c, k, ha, hb);
    const float2 xa = buf[ia], xb = buf[ib];
    buf[ia] = pair_product(xa, xb, ha, hb);
    if (ib != ia) buf[ib] = pair_product(xb, xa, conjf2(ha), conjf2(hb));
  };
  const int npairs = gi == 0 ? (N1 / 2 + 1 + N1 / 2) * WCM : N1 * G * WCM;
  for (int u = (int)threadIdx.x; u < npairs; u += NT) {
    const int cc = u % WCM, r = u / WCM;
    const int x = x0 + cc;
    if (x >= ch.nvalid) continue;
    const int g = ch.g0 + x;
    const int m = g / ch.ncc;
    const int c = 2 * (g - m * ch.ncc);
    if (gi == 0) {
      if (r <= N1 / 2) {  // k2 = 0: bins N2 k1 and N2 ((N1 - k1) mod N1)
        const int k1 = r, pk1 = (N1 - k1) & (N1 - 1);
        pair(k1 * W + cc, pk1 * W + cc, N2 * k1, m, c);
      } else {            // k2 = N2/2: bins N2 k1 + N2/2 and its mirror at N1-1-k1
        const int k1 = r - (N1 / 2 + 1), pk1 = N1 - 1 - k1;
        pair(k1 * W + WCM + cc, pk1 * W + WCM + cc, N2 * k1 + N2 / 2, m, c);
      }
    } else {
      const int s = r % G, k1 = r / G;
      const int k2 = mid_slot_k2(gi, s, N2);
      if (k2 < 0) continue;
      pair(k1 * W + s * WCM + cc, (N1 - 1 - k1) * W + (G + s) * WCM + cc, N2 * k1 + k2, m, c);
    }
  }
  __syncthreads();
  fft::lds_passes<N1, 0, fft::Plan<N1>::NP, W, W, NT, true>(buf, twz);
  for (int u = (int)threadIdx.x; u < N1 * W; u += NT) {
    const int n1 = u / W, slot = (u - n1 * W) / WCM, cc = u % WCM;
    const int k2 = mid_slot_k2(gi, slot, N2);
    const int x = x0 + cc;
    if (k2 < 0 || x >= ch.nvalid) continue;
    C[(size_t)(n1 * N2 + k2) * ch.cstride + x] = cmulc(buf[u], fft::twiddle<false>(tw, N, n1 * k2));
  }
}

// Pass R': inverse N2-point FFT of E[n1][.] for each n1; output n2 >= N2/2 is
// time index n = n1 + N1 n2 >= U and is added into state row i + n - U when
// n - U < dst_len.  STORE: stored into row i - U + n - U instead (over the
// inputs, which the chunk's first pass has read).
template <int N2, bool STORE>
__global__ __launch_bounds__(Cfg<N2>::NT) void k_fft_rows_inv(const float2* __restrict__ E,
                                                              float* __restrict__ S, int SL, int i,
                                                              int dst_len, Chunk ch,
                                                              const float2* __restrict__ tw) {
  constexpr int WC = Cfg<N2>::WC, NT = Cfg<N2>::NT;
  using P = fft::Plan<N2>;
  __shared__ float2 buf[N2 * WC];
  __shared__ float2 twl[Cfg<N2>::TWN];
  const auto twz = make_tw<N2>(twl, tw);
  const int npan = (ch.nvalid + WC - 1) / WC;
  const int q = fft::xcd_logical((int)blockIdx.x, (int)gridDim.x);
  const int n1 = q / npan;
  const int x0 = (q - n1 * npan) * WC;
  const int N1 = ch.N1, U = N1 * N2 / 2, BD = ch.ncols;
  const bool vec = (BD & 1) == 0;
  for (int u = (int)threadIdx.x; u < N2 * WC; u += NT) {
    const int k2 = u / WC, col = u - k2 * WC;
    const int x = x0 + col;
    buf[u] = x < ch.nvalid ? E[(size_t)(n1 * N2 + k2) * ch.cstride + x] : make_float2(0.f, 0.f);
  }
  // destination rows of the last pass (radix RL, p = N2/RL): unit j writes
  // n2 = j + s N2/RL for s >= RL/2, time index n1 + N1 n2 = U + n1 + N1 (j + (s - RL/2) PL)
  constexpr int RL = P::radix(P::NP - 1);
  constexpr int PL = N2 / RL;
  constexpr int LUN = PL * WC;
  constexpr int LU = (LUN + NT - 1) / NT;
  float* rowp[LU];  // row of output 0 in the column's layer, nullptr for no column
  int cpos[LU];     // real column index of the pair
  float2 zo[LU][RL / 2];
#pragma unroll
  for (int a = 0; a < LU; ++a) {
    const int u = (int)threadIdx.x + a * NT;
    const int j = u / WC, col = u - j * WC;
    const int x = x0 + col;
    rowp[a] = nullptr;
    cpos[a] = 0;
    if (u < LUN && x < ch.nvalid) {
      const int g = ch.g0 + x;
      const int m = g / ch.ncc;
      rowp[a] = S + ((size_t)m * SL + (STORE ? i - U : i)) * BD;
      cpos[a] = 2 * (g - m * ch.ncc);
    }
#pragma unroll
    for (int s = 0; s < RL / 2; ++s) {
      const int oi = n1 + N1 * (j + s * PL);
      zo[a][s] = (!STORE && rowp[a] && oi < dst_len)
                     ? load_pair(rowp[a] + (size_t)oi * BD, cpos[a], BD, vec)
                     : make_float2(0.f, 0.f);
    }
  }
  __syncthreads();
  fft::lds_passes<N2, 0, P::NP - 1, WC, WC, NT, true>(buf, twz);
#pragma unroll
  for (int a = 0; a < LU; ++a) {
    const int u = (int)threadIdx.x + a * NT;
    if (u < LUN && rowp[a]) {
      const int j = u / WC, col = u - j * WC;  // j < PL, so k = j
      float2 v[RL];
#pragma unroll
      for (int t = 0; t < RL; ++t) v[t] = buf[(j + t * PL) * WC + col];
      if constexpr (PL > 1) {
#pragma unroll
        for (int t = 1; t < RL; ++t) v[t] = cmul(v[t], twz.template get<true, N2>(t * j));
      }
      fft::dft<RL, true>(v);
      const int c = cpos[a];
      (void)col;
#pragma unroll
      for (int s = 0; s < RL / 2; ++s) {
        const int oi = n1 + N1 * (j + s * PL);
        if (oi < dst_len) {
          float* row = rowp[a] + (size_t)oi * BD;
          const float2 o = STORE ? v[RL / 2 + s]
                                 : make_float2(zo[a][s].x + v[RL / 2 + s].x,
                                               zo[a][s].y + v[RL / 2 + s].y);
          if (vec) {
            *reinterpret_cast<float2*>(row + c) = o;
          } else {
            row[c] = o.x;
            if (c + 1 < BD) row[c + 1] = o.y;
          }
        }
      }
    }
  }
}

// ------------------------------------------------------------- dispatch

#define LCSM_POW2_CASES(X) \
  X(4) X(8) X(16) X(32) X(64) X(128) X(256) X(512) X(1024) X(2048) X(4096) X(8192)

// Panel width WC of the single-pass tiles is Cfg<N>::WC, except at 2U = 128
// and 256 when the launch has many columns: there 8-column panels (64-byte
// row runs instead of 32) take the tile 25 % faster at 55K and 1M columns,
// while at a few thousand columns the halved workgroup count leaves CUs idle.
constexpr int kWideWC = 8;

template <int NN, int WC>
hipError_t tile_panels(float* S, const float2* H, const float2* tw, const float* Hf,
                       const float* yt, float* zt, const Shape& s, int i, int dst_len,
                       bool in_place, hipStream_t st) {
  const int ppl = (s.BD + 2 * WC - 1) / (2 * WC);
  const int hgroup = (s.D % (2 * WC) == 0) ? s.D / (2 * WC) : 0;
  const dim3 grid((unsigned)(ppl * s.M)), block(Cfg<NN>::NT);
  const bool fast = hgroup > 0 && dst_len == NN / 2;
#define LCSM_TILE(RED, FAST, STORE)                                                          \
  hipLaunchKernelGGL((k_fft_tile<NN, RED, FAST, STORE, WC>), grid, block, 0, st, S, H, tw, Hf, \
                     yt, zt, s.L, s.SL, s.BD, s.D, s.B, i, dst_len, ppl, hgroup)
  if (yt) {
    if constexpr (NN <= kMaxRedFftN) {
      if (fast)
        LCSM_TILE(true, true, false);
      else
        LCSM_TILE(true, false, false);
    } else {
      return hipErrorInvalidValue;
    }
  } else if (in_place) {
    if (fast)
      LCSM_TILE(false, true, true);
    else
      LCSM_TILE(false, false, true);
  } else if (fast) {
    LCSM_TILE(false, true, false);
  } else {
    LCSM_TILE(false, false, false);
  }
#undef LCSM_TILE
  return hipGetLastError();
}

hipError_t tile_single(int N, float* S, const float2* H, const float2* tw, const float* Hf,
                       const float* yt, float* zt, const Shape& s, int i, int dst_len,
                       bool in_place, hipStream_t st) {
  const bool wide = (long long)s.M * s.BD >= kWidePanelMinCols;
#define LCSM_CASE(NN)                                                                      \
  case NN:                                                                                 \
    if constexpr (NN == 128 || NN == 256) {                                                \
      if (wide)                                                                            \
        return tile_panels<NN, kWideWC>(S, H, tw, Hf, yt, zt, s, i, dst_len, in_place, st); \
    }                                                                                      \
    return tile_panels<NN, Cfg<NN>::WC>(S, H, tw, Hf, yt, zt, s, i, dst_len, in_place, st);
  switch (N) { LCSM_POW2_CASES(LCSM_CASE) }
#undef LCSM_CASE
  return hipErrorInvalidValue;
}

hipError_t spectra_single(int N, const float* Hf, float2* Hout, const float2* tw, const Shape& s,
                          int shift, int colmaj, hipStream_t st) {
#define LCSM_CASE(NN)                                                                            \
  case NN: {                                                                                     \
    const int ppl = (s.D + 2 * Cfg<NN>::WC - 1) / (2 * Cfg<NN>::WC);                             \
    hipLaunchKernelGGL(k_fft_spectra<NN>, dim3((unsigned)(ppl * s.M)), dim3(Cfg<NN>::NT), 0, st, \
                       Hf, Hout, tw, s.L, s.D, ppl, shift, colmaj);                                      \
    return hipGetLastError();                                                                    \
  }
  switch (N) { LCSM_POW2_CASES(LCSM_CASE) }
#undef LCSM_CASE
  return hipErrorInvalidValue;
}

#define LCSM_ROW_CASES(X) X(16) X(32) X(64) X(128) X(256) X(512) X(1024) X(2048) X(4096)
#define LCSM_MID_CASES(X) X(2) X(4) X(8) X(16) X(32) X(64) X(128)

template <bool HALF>
hipError_t rows_fwd(const float* src, size_t lstride, int row0, int rows_valid, const Chunk& ch,
                    float2* C, const float2* tw, hipStream_t st) {
#define LCSM_CASE(NN)                                                                            \
  case NN: {                                                                                     \
    const int npan = (ch.nvalid + Cfg<NN>::WC - 1) / Cfg<NN>::WC;                                \
    hipLaunchKernelGGL((k_fft_rows_fwd<NN, HALF>), dim3((unsigned)(npan * ch.N1)),               \
                       dim3(Cfg<NN>::NT), 0, st, src, lstride, row0, rows_valid, ch, C, tw);     \
    return hipGetLastError();                                                                    \
  }
  switch (ch.N2) { LCSM_ROW_CASES(LCSM_CASE) }
#undef LCSM_CASE
  return hipErrorInvalidValue;
}

template <bool STORE>
hipError_t rows_inv(const float2* E, float* S, int SL, int i, int dst_len, const Chunk& ch,
                    const float2* tw, hipStream_t st) {
#define LCSM_CASE(NN)                                                                           \
  case NN: {                                                                                    \
    const int npan = (ch.nvalid + Cfg<NN>::WC - 1) / Cfg<NN>::WC;                               \
    hipLaunchKernelGGL((k_fft_rows_inv<NN, STORE>), dim3((unsigned)(npan * ch.N1)),             \
                       dim3(Cfg<NN>::NT), 0, st, E, S, SL, i, dst_len, ch, tw);                 \
    return hipGetLastError();                                                                   \
  }
  switch (ch.N2) { LCSM_ROW_CASES(LCSM_CASE) }
#undef LCSM_CASE
  return hipErrorInvalidValue;
}

hipError_t mid_tile(float2* C, const float2* H, int D, const Chunk& ch, const float2* tw,
                    hipStream_t st) {
  const int npan = (ch.nvalid + kMidWC - 1) / kMidWC;
  const int groups = 1 + (ch.N2 / 2 - 1 + kMidG - 1) / kMidG;
  const dim3 grid((unsigned)(npan * groups));
#define LCSM_CASE(NN)                                                                           \
  case NN:                                                                                      \
    hipLaunchKernelGGL(k_fft_mid_tile<NN>, grid, dim3(kMidNT), 0, st, C, H, D, ch, tw);         \
    return hipGetLastError();
  switch (ch.N1) { LCSM_MID_CASES(LCSM_CASE) }
#undef LCSM_CASE
  return hipErrorInvalidValue;
}

hipError_t mid_spectra(const float2* C, float2* Hout, int D, const Chunk& ch, const float2* tw,
                       int colmaj, hipStream_t st) {
  const int npan = (ch.nvalid + kMidWC - 1) / kMidWC;
  const dim3 grid((unsigned)(npan * (ch.N2 / kMidG)));
#define LCSM_CASE(NN)                                                                             \
  case NN:                                                                                        \
    hipLaunchKernelGGL(k_fft_mid_spectra<NN>, grid, dim3(kMidNT), 0, st, C, Hout, D, ch, tw, colmaj);     \
    return hipGetLastError();
  switch (ch.N1) { LCSM_MID_CASES(LCSM_CASE) }
#undef LCSM_CASE
  return hipErrorInvalidValue;
}

// Row length of the multi-pass split of an N-point transform: 1024-point
// rows (four row workgroups per CU) measured fastest while the columns stay
// short; 4096-point rows when the columns would be longer than
// kPreferredMidN1 points (a 128-point column pass runs at one wave per SIMD).
int split_n2(int N, int lds_max_n) {
  int n2 = lds_max_n < kPreferredRowN2 ? lds_max_n : kPreferredRowN2;
  while (N / n2 > kMaxMidN1) n2 *= 2;
  // past the preferred column length, straight to the longest rows (2048-point
  // rows measured slower than both 1024- and 4096-point ones)
  if (N / n2 > kPreferredMidN1 && N / kMaxRowN2 >= 2 && n2 < kMaxRowN2) n2 = kMaxRowN2;
  return n2;
}

}  // namespace

int fft_multipass_chunk(int N, size_t scratch_bytes, int total_cc) {
  // one N-point complex column of C per chunk column (pass M works in place)
  long long cap = (long long)(scratch_bytes / (sizeof(float2) * (size_t)N));
  cap = cap / 16 * 16;
  const long long need = ((long long)total_cc + 15) / 16 * 16;
  if (cap > need) cap = need;
  return (int)cap;
}

hipError_t launch_spectra(const float* Hf, float2* Hout, const float2* tw, const Shape& s, int U,
                          int shift, int lds_max_n, float2* scratch, size_t scratch_bytes,
                          hipStream_t st, bool colmaj) {
  const int N = 2 * U;
  if (N <= lds_max_n) return spectra_single(N, Hf, Hout, tw, s, shift, colmaj ? 1 : 0, st);
  Chunk ch{};
  ch.ncols = s.D;
  ch.ncc = (s.D + 1) / 2;
  ch.N2 = split_n2(N, lds_max_n);
  ch.N1 = N / ch.N2;
  const int total = s.M * ch.ncc;
  ch.cstride = fft_multipass_chunk(N, scratch_bytes, total);
  if (ch.cstride <= 0) return hipErrorOutOfMemory;
  float2* C = scratch;
  for (int g0 = 0; g0 < total; g0 += ch.cstride) {
    ch.g0 = g0;
    ch.nvalid = total - g0 < ch.cstride ? total - g0 : ch.cstride;
    hipError_t e = rows_fwd<false>(Hf, (size_t)s.L * s.D, -shift, s.L, ch, C, tw, st);
    if (e == hipSuccess) e = mid_spectra(C, Hout, s.D, ch, tw, colmaj ? 1 : 0, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_fft_tile(float* S, const float2* H, const float2* tw, const Shape& s, int i,
                           int U, int dst_len, int lds_max_n, float2* scratch, size_t scratch_bytes,
                           hipStream_t st, bool in_place) {
  if (dst_len <= 0) return hipSuccess;
  const int N = 2 * U;
  if (N <= lds_max_n)
    return tile_single(N, S, H, tw, nullptr, nullptr, nullptr, s, i, dst_len, in_place, st);
  Chunk ch{};
  ch.ncols = s.BD;
  ch.ncc = (s.BD + 1) / 2;
  ch.N2 = split_n2(N, lds_max_n);
  ch.N1 = N / ch.N2;
  const int total = s.M * ch.ncc;
  ch.cstride = fft_multipass_chunk(N, scratch_bytes, total);
  if (ch.cstride <= 0) return hipErrorOutOfMemory;
  float2* C = scratch;
  for (int g0 = 0; g0 < total; g0 += ch.cstride) {
    ch.g0 = g0;
    ch.nvalid = total - g0 < ch.cstride ? total - g0 : ch.cstride;
    // the chunk's columns: all inputs into C, then (stream order) the outputs
    hipError_t e = rows_fwd<true>(S, (size_t)s.SL * s.BD, i - U, i, ch, C, tw, st);
    if (e == hipSuccess) e = mid_tile(C, H, s.D, ch, tw, st);
    if (e == hipSuccess)
      e = in_place ? rows_inv<true>(C, S, s.SL, i, dst_len, ch, tw, st)
                   : rows_inv<false>(C, S, s.SL, i, dst_len, ch, tw, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_red_fft_tile(const float* yt, float* zt, float* S, const float* Hf,
                               const float2* H, const float2* tw, const Shape& s, int i, int U,
                               int dst_len, hipStream_t st) {
  return tile_single(2 * U, S, H, tw, Hf, yt, zt, s, i, dst_len, false, st);
}

}  // namespace lcsm
