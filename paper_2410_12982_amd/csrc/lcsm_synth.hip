// The synthetic end-to-end model of the experiments (Sec. 5): per layer a
// long-convolution mixer and an MLP block of hidden width 2D with the exact
// GELU; the next token's input is the last layer's output plus noise (the
// sampler of Alg. 3).
//
// Per position t the work is (all on the mixer context's stream):
//   k_synth_red0            y^0_t = eps_t (+ a^M_{t-1}); layer 0's red cell
//   for each layer m:
//     k_gemv<UP>            hid = gelu(W_up[m] z^m_t + b_up[m])        [B][2D]
//     k_gemv<DOWN>          a^{m+1}_t = W_down[m] hid + b_down[m] -> act[m];
//                           its epilogue is layer m+1's red cell (y^{m+1}_t =
//                           a^{m+1}_t), or keeps a^M_t for the sampler
//   the gray tiles of i = t+1 for all layers (the mixer's batched launch).
//
// The products are matrix-vector products over B <= 16 rows at a time: their
// time is the weight read (4 bytes per weight, 2B flops).  Small ones are
// bound by how many loads are in flight, not by bytes: a workgroup takes one
// output unit and splits its weight row over K/256 waves, one 1 KB piece per
// wave (its 64 lanes in 16-byte parts), multiplied with the same pieces of
// the B input rows; each wave reduces with butterfly shuffles and wave 0 sums
// the waves' partials from LDS in wave order (deterministic), after which
// lane r stores row r.  With 8 and more rows against large weight matrices
// that form is bound by re-reading the input rows for every unit, and the
// products take the matrix cores instead (k_gemm16: 16 units per
// workgroup, the 16 x 16 block of rows and units accumulated in four
// registers per lane), which read the inputs once per 16 units.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <new>

#include "lcsm_internal.h"
#include "lcsm_synth.h"

namespace lcsm {
namespace {

constexpr int kGemvMaxThreads = 1024;  // 16 waves: K up to 4096 in one piece per wave
constexpr int kMaxRows = 16;     // batch rows per product launch

enum { kUp = 0, kDown = 1 };

// Arguments of the DOWN epilogue: the next layer's red cell, or the copy of
// a^M_t for the sampler (S == nullptr).
struct RedNext {
  float* S;          // state slot row of position t, layer m+1: S + (m+1)*SL*BD + t*BD
  const float* h0;   // filter taps h[m+1, d, 0] (lag-0 row of layer m+1)
  float* z;          // [B][D] the next layer's mixer output
  float* last;       // [B][D] a^M_t (last layer only)
};

__device__ __forceinline__ float gelu(float v) {
  return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
}

// out rows r < nrows of the product W [N][K] x^T with x [nrows][K] (row
// stride K): MODE kUp -> out[r][n] = gelu(sum + bias[n]) (row stride N);
// MODE kDown -> a = sum + bias[n], out[r][n] = a (row stride N = D), then the
// red cell of the next layer or the sampler copy.  NR >= nrows, a power of
// two <= kMaxRows; rows nrows..NR-1 are computed from row nrows-1 and not
// stored.  K must be a multiple of 4 and the rows 16-byte aligned.
// One output unit per workgroup: its WPU waves take consecutive 256-float
// pieces of the unit's weight row (wave w: pieces w, w + WPU, ...), reduce
// over the wave with butterfly shuffles, and wave 0 sums the WPU partials of
// each row from LDS (in wave order: deterministic).
template <int NR, int MODE>
__global__ __launch_bounds__(kGemvMaxThreads) void k_gemv(const float* __restrict__ x,
                                                          const float* __restrict__ W,
                                                          const float* __restrict__ bias,
                                                          float* __restrict__ out, int N, int K,
                                                          int nrows, RedNext rn) {
  __shared__ float part[kGemvMaxThreads / 64][NR];
  const int lane = (int)threadIdx.x & 63, wv = (int)threadIdx.x >> 6;
  const int wpu = (int)blockDim.x >> 6;
  const int n = (int)blockIdx.x;
  const float* wr = W + (size_t)n * K;
  const float* xr[NR];
#pragma unroll
  for (int r = 0; r < NR; ++r) xr[r] = x + (size_t)(r < nrows ? r : nrows - 1) * K;
  float acc[NR];
#pragma unroll
  for (int r = 0; r < NR; ++r) acc[r] = 0.f;
  for (int k = wv * 256 + lane * 4; k < K; k += wpu * 256) {
    const float4 w = *reinterpret_cast<const float4*>(wr + k);
    float4 v[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) v[r] = *reinterpret_cast<const float4*>(xr[r] + k);
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      acc[r] = fmaf(w.x, v[r].x, acc[r]);
      acc[r] = fmaf(w.y, v[r].y, acc[r]);
      acc[r] = fmaf(w.z, v[r].z, acc[r]);
      acc[r] = fmaf(w.w, v[r].w, acc[r]);
    }
  }
#pragma unroll
  for (int r = 0; r < NR; ++r) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) acc[r] += __shfl_xor(acc[r], off, 64);
  }
  if (lane < NR) {
#pragma unroll
    for (int r = 0; r < NR; ++r)
      if (r == lane) part[wv][r] = acc[r];
  }
  __syncthreads();
  if (wv != 0 || lane >= nrows) return;
  const int r = lane;
  float s = 0.f;
  for (int q = 0; q < wpu; ++q) s += part[q][r];
  s += bias[n];
  const size_t e = (size_t)r * N + n;
  if constexpr (MODE == kUp) {
    out[e] = gelu(s);
  } else {
    out[e] = s;
    if (rn.S) {
      float* slot = rn.S + e;
      rn.z[e] = fmaf(rn.h0[n], s, *slot);
      *slot = s;
    } else {
      rn.last[e] = s;
    }
  }
}

// The same product on the matrix cores, for several batch rows: a
// workgroup takes 16 output units (or 8, with the block's other 8 columns
// repeating them, where 16 would leave compute units idle) and splits K over
// its waves; each wave
// accumulates the 16 x 16 block (rows x units) of its K-slice with
// v_mfma_f32_16x16x4f32, 16 k per step (lane l loads 4 consecutive k of
// unit n0 + l%16 and of row l%16 at offset 4 (l/16); the four products of a
// step take the four components, the same k on both operands).  The input
// rows are then read once per 16 units instead of once per unit, and no
// lane reductions are needed.  The waves' blocks are summed from LDS in
// wave order (deterministic), then the same epilogue as k_gemv.  Rows past
// nrows and units past N load clamped rows and are not stored; K is a
// multiple of 4.
typedef float v4f __attribute__((ext_vector_type(4)));

template <int MODE>
__global__ __launch_bounds__(kGemvMaxThreads) void k_gemm16(const float* __restrict__ x,
                                                            const float* __restrict__ W,
                                                            const float* __restrict__ bias,
                                                            float* __restrict__ out, int N, int K,
                                                            int nrows, int ut, RedNext rn) {
  __shared__ float part[kGemvMaxThreads / 64][256];
  const int lane = (int)threadIdx.x & 63, wv = (int)threadIdx.x >> 6;
  const int nw = (int)blockDim.x >> 6;
  const int n0 = (int)blockIdx.x * ut;  // ut = 16 units per workgroup, or 8 (columns 8..15 repeat them)
  const int j = lane & 15, q = lane >> 4;
  const int ju = j < ut ? j : j - ut;
  const int un = n0 + ju < N ? n0 + ju : N - 1;  // unit whose weights this lane loads
  const int xr = j < nrows ? j : nrows - 1;     // batch row whose inputs this lane loads
  const float* wrow = W + (size_t)un * K + 4 * q;
  const float* xrow = x + (size_t)xr * K + 4 * q;
  // the wave's k-blocks of 16: a contiguous range
  const int nkb = (K + 15) / 16;
  const int per = (nkb + nw - 1) / nw;
  const int kb0 = wv * per, kb1 = kb0 + per < nkb ? kb0 + per : nkb;
  v4f acc = {0.f, 0.f, 0.f, 0.f};
  // four k-blocks' loads in flight, then their 16 products
  for (int kb = kb0; kb < kb1; kb += 4) {
    float4 wf[4], xf[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int k = 16 * (kb + u);
      wf[u] = xf[u] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (kb + u < kb1 && k + 4 * q < K) {
        wf[u] = *reinterpret_cast<const float4*>(wrow + k);
        xf[u] = *reinterpret_cast<const float4*>(xrow + k);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(xf[u].x, wf[u].x, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(xf[u].y, wf[u].y, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(xf[u].z, wf[u].z, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(xf[u].w, wf[u].w, acc, 0, 0, 0);
    }
  }
  // lane (jj + 16 g) holds rows 4g .. 4g+3 of unit column jj
#pragma unroll
  for (int v = 0; v < 4; ++v) part[wv][(4 * q + v) * 16 + j] = acc[v];
  __syncthreads();
  for (int o = (int)threadIdx.x; o < 256; o += (int)blockDim.x) {
    const int r = o >> 4, n = n0 + (o & 15);
    if (r >= nrows || (o & 15) >= ut || n >= N) continue;
    float sacc = 0.f;
    for (int w = 0; w < nw; ++w) sacc += part[w][o];
    const float sv = sacc + bias[n];
    const size_t e = (size_t)r * N + n;
    if constexpr (MODE == kUp) {
      out[e] = gelu(sv);
    } else {
      out[e] = sv;
      if (rn.S) {
        float* slot = rn.S + e;
        rn.z[e] = fmaf(rn.h0[n], sv, *slot);
        *slot = sv;
      } else {
        rn.last[e] = sv;
      }
    }
  }
}

// Sampler and layer 0's red cell at position t: y = eps (+ last for t > 0),
// z = fmaf(h0[d], y, slot), slot = y.
__global__ __launch_bounds__(256) void k_synth_red0(const float* __restrict__ eps,
                                                    const float* __restrict__ last,
                                                    float* __restrict__ slot_row,
                                                    const float* __restrict__ h0,
                                                    float* __restrict__ z, int BD, int D, int t) {
  const int c = (int)blockIdx.x * 256 + (int)threadIdx.x;
  if (c >= BD) return;
  const float y = t > 0 ? last[c] + eps[c] : eps[c];
  z[c] = fmaf(h0[c % D], y, slot_row[c]);
  slot_row[c] = y;
}

// Which form a product takes.  The matrix-core form reads the input rows
// once per 16 units, which pays where the per-unit form is bound by those
// reads (8 and more rows against large weight matrices: 16 rows x 2048 x
// 4096 ran 3.1x faster); on the latency-bound small products of 4 and 8 rows
// x 768 it was 4-37 % slower (fewer waves in flight).
inline bool gemm16_for(int N, int K, int nrows) {
  return nrows >= 8 && (int64_t)N * K >= ((int64_t)1 << 22);
}

template <int MODE>
hipError_t gemv(const float* x, const float* W, const float* bias, float* out, int N, int K,
                int nrows, const RedNext& rn, hipStream_t st) {
  if (gemm16_for(N, K, nrows)) {
    // 16 units per workgroup, about four k-blocks of 16 per wave, at most 16 waves
    int nw = (K + 63) / 64;
    if (nw > kGemvMaxThreads / 64) nw = kGemvMaxThreads / 64;
    if (nw < 1) nw = 1;
    // 8 units per workgroup where 16 would leave CUs idle (the column blocks
    // 8..15 then repeat units 0..7 and are not stored)
    const int ut = (N + 15) / 16 >= 256 ? 16 : 8;
    hipLaunchKernelGGL((k_gemm16<MODE>), dim3((unsigned)((N + ut - 1) / ut)),
                       dim3((unsigned)(64 * nw)), 0, st, x, W, bias, out, N, K, nrows, ut, rn);
    return hipGetLastError();
  }
  int wpu = (K + 255) / 256;  // waves per unit: one 256-float piece each
  if (wpu > kGemvMaxThreads / 64) wpu = kGemvMaxThreads / 64;
  const dim3 grid((unsigned)N), block((unsigned)(64 * wpu));
#define LCSM_GEMV(NR) \
  hipLaunchKernelGGL((k_gemv<NR, MODE>), grid, block, 0, st, x, W, bias, out, N, K, nrows, rn)
  if (nrows <= 1)
    LCSM_GEMV(1);
  else if (nrows <= 2)
    LCSM_GEMV(2);
  else if (nrows <= 4)
    LCSM_GEMV(4);
  else if (nrows <= 8)
    LCSM_GEMV(8);
  else
    LCSM_GEMV(16);
#undef LCSM_GEMV
  return hipGetLastError();
}

}  // namespace
}  // namespace lcsm

struct lcsm_synth {
  lcsm_ctx* mixer;
  int M, B, D, L;
  hipStream_t stream;
  char* mem;
  float *w_up, *b_up, *w_down, *b_down;
  float *z, *hid, *last;
  bool faulted;
  char msg[256];
};

namespace {

int synth_fail(lcsm_synth* s, int code, const char* what, hipError_t e) {
  if (e != hipSuccess) {
    snprintf(s->msg, sizeof(s->msg), "%s: %s", what, hipGetErrorString(e));
    s->faulted = true;
    return LCSM_EDEVICE;
  }
  snprintf(s->msg, sizeof(s->msg), "%s", what);
  return code;
}

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

}  // namespace

extern "C" {

int lcsm_synth_init(lcsm_synth** out, const float* filters, const float* w_up, const float* b_up,
                    const float* w_down, const float* b_down, int M, int B, int D, int L,
                    void* stream, const lcsm_options* opt) {
  if (!out) return LCSM_EINVAL;
  *out = nullptr;
  if (!filters || !w_up || !b_up || !w_down || !b_down) return LCSM_EINVAL;
  if (D < 4 || D % 4 != 0) return LCSM_EINVAL;
  size_t need = 0;
  int r = lcsm_workspace_bytes(M, B, D, L, opt, &need);  // validates shape and options
  if (r) return r;
  lcsm_synth* s = new (std::nothrow) lcsm_synth();
  if (!s) return LCSM_ENOMEM;
  s->M = M;
  s->B = B;
  s->D = D;
  s->L = L;
  s->stream = (hipStream_t)stream;
  s->msg[0] = 0;
  const size_t D2 = 2 * (size_t)D, BD = (size_t)B * D;
  const size_t n_wup = (size_t)M * D2 * D, n_bup = (size_t)M * D2, n_wdn = (size_t)M * D * D2,
               n_bdn = (size_t)M * D;
  size_t off[7], total = 0;
  const size_t sizes[7] = {n_wup, n_bup, n_wdn, n_bdn, BD, (size_t)B * D2, BD};
  for (int k = 0; k < 7; ++k) {
    off[k] = total;
    total = align256(total + sizeof(float) * sizes[k]);
  }
  void* p = nullptr;
  if (hipMalloc(&p, total) != hipSuccess) {
    (void)hipGetLastError();
    delete s;
    return LCSM_ENOMEM;
  }
  s->mem = (char*)p;
  float* f[7];
  for (int k = 0; k < 7; ++k) f[k] = (float*)(s->mem + off[k]);
  s->w_up = f[0];
  s->b_up = f[1];
  s->w_down = f[2];
  s->b_down = f[3];
  s->z = f[4];
  s->hid = f[5];
  s->last = f[6];
  r = lcsm_init(&s->mixer, filters, M, B, D, L, stream, nullptr, 0, opt);
  if (r) {
    (void)hipFree(s->mem);
    delete s;
    return r;
  }
  const float* src[4] = {w_up, b_up, w_down, b_down};
  hipError_t e = hipSuccess;
  for (int k = 0; k < 4 && e == hipSuccess; ++k)
    e = hipMemcpyAsync(f[k], src[k], sizeof(float) * sizes[k], hipMemcpyDeviceToDevice, s->stream);
  if (e == hipSuccess) e = lcsm::launch_zero(s->last, BD, s->stream);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    lcsm_destroy(s->mixer);
    (void)hipFree(s->mem);
    delete s;
    return LCSM_EDEVICE;
  }
  s->faulted = false;
  *out = s;
  return LCSM_OK;
}

int lcsm_synth_step(lcsm_synth* s, const float* eps_t, float* act_t) {
  if (!s) return LCSM_EINVAL;
  if (!eps_t || !act_t) return synth_fail(s, LCSM_EINVAL, "null input or output pointer", hipSuccess);
  if (s->faulted) return LCSM_ESTATE;
  lcsm::StepView v;
  int r = lcsm::begin_external_step(s->mixer, &v);
  if (r) return r == LCSM_EDONE ? r : synth_fail(s, r, lcsm_last_error(s->mixer), hipSuccess);
  const int M = s->M, B = s->B, D = s->D, D2 = 2 * D, BD = B * D;
  const size_t lstride = (size_t)v.s.SL * BD;  // state floats per layer
  const size_t hstride = (size_t)v.s.L * D;    // filter floats per layer
  hipStream_t st = v.stream;
  // sampler + layer 0's red cell (state slot row of position t, layer 0)
  hipLaunchKernelGGL(lcsm::k_synth_red0, dim3((unsigned)((BD + 255) / 256)), dim3(256), 0, st,
                     eps_t, s->last, v.S + (size_t)v.t * BD, v.Hf, s->z, BD, D, v.t);
  hipError_t e = hipGetLastError();
  for (int m = 0; m < M && e == hipSuccess; ++m) {
    for (int r0 = 0; r0 < B && e == hipSuccess; r0 += lcsm::kMaxRows) {
      const int nr = B - r0 < lcsm::kMaxRows ? B - r0 : lcsm::kMaxRows;
      lcsm::RedNext none{nullptr, nullptr, nullptr, nullptr};
      e = lcsm::gemv<lcsm::kUp>(s->z + (size_t)r0 * D, s->w_up + (size_t)m * D2 * D,
                                s->b_up + (size_t)m * D2, s->hid + (size_t)r0 * D2, D2, D, nr,
                                none, st);
      lcsm::RedNext rn{nullptr, nullptr, nullptr, nullptr};
      if (m + 1 < M) {
        rn.S = v.S + (size_t)(m + 1) * lstride + (size_t)v.t * BD + (size_t)r0 * D;
        rn.h0 = v.Hf + (size_t)(m + 1) * hstride;
        rn.z = s->z + (size_t)r0 * D;
      } else {
        rn.last = s->last + (size_t)r0 * D;
      }
      if (e == hipSuccess)
        e = lcsm::gemv<lcsm::kDown>(s->hid + (size_t)r0 * D2, s->w_down + (size_t)m * D * D2,
                                    s->b_down + (size_t)m * D,
                                    act_t + (size_t)m * BD + (size_t)r0 * D, D, D2, nr, rn, st);
    }
  }
  if (e != hipSuccess) return synth_fail(s, LCSM_EDEVICE, "model kernel launch", e);
  r = lcsm::end_external_step(s->mixer);
  if (r) return synth_fail(s, r, lcsm_last_error(s->mixer), hipSuccess);
  return LCSM_OK;
}

int lcsm_synth_reset(lcsm_synth* s) {
  if (!s) return LCSM_EINVAL;
  int r = lcsm_reset(s->mixer);
  if (r) return synth_fail(s, r, lcsm_last_error(s->mixer), hipSuccess);
  s->faulted = false;
  s->msg[0] = 0;
  return LCSM_OK;
}

int lcsm_synth_position(const lcsm_synth* s, int* t) {
  if (!s || !t) return LCSM_EINVAL;
  return lcsm_position(s->mixer, t);
}

void lcsm_synth_destroy(lcsm_synth* s) {
  if (!s) return;
  lcsm_destroy(s->mixer);  // waits for the stream
  (void)hipFree(s->mem);
  delete s;
}

const char* lcsm_synth_last_error(const lcsm_synth* s) { return s ? s->msg : ""; }

}  // extern "C"
