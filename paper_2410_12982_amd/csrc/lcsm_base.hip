// Lazy and eager online convolutions (the baselines of Sec. 3.1.1 and
// Sec. 5), for gfx950.
//
// Layout as in the relaxed library: state S[m][t][c] with c = b*D + d
// (time-major), filters Hf[m][k][d] (lag-major).  A thread owns one column
// of one layer for a range of positions; consecutive threads take
// consecutive columns, so every row access of a wavefront is one contiguous
// run.  The batch rows of a layer read the same filter rows.
//
// Lazy step t: z_t = fmaf(h_0, y_t, sum_{s<t} y_s h_{t-s}).  The sum over s
// is split into chunks of kLazyCh positions, one workgroup per chunk and
// column block (k_lazy_partial), and the partial sums are added in chunk
// order by k_lazy_reduce, which also stores y_t into the state: the sum is
// the same fixed-order one on every run.  Up to kLazyCh earlier positions
// one kernel does all of it (k_lazy_fused).
//
// Eager step t: z_t = fmaf(h_0, y_t, acc_t); acc_r = fmaf(y_t, h_{r-t},
// acc_r) for r = t+1 .. L-1, split into chunks of kEagerCh rows
// (k_eager_step; chunk 0's workgroups also emit z_t).  Each accumulator is
// updated once per step, in step order.
#include <stdio.h>

#include <new>

#include "lcsm_base.h"
#include "lcsm_internal.h"

namespace lcsm {
namespace {

constexpr int kBT = 256;        // threads per workgroup (columns)
constexpr int kLazyCh = 256;    // positions per partial sum
constexpr int kEagerCh = 64;    // accumulator rows per workgroup
constexpr int kUnroll = 8;      // loads in flight per thread and loop step

inline unsigned col_blocks(int BD) { return (unsigned)((BD + kBT - 1) / kBT); }

// sum_{s in [s0, s1)} y_s h_{t-s} for column c of layer m, in increasing s
// with kUnroll independent accumulators combined pairwise at the end.
__device__ __forceinline__ float lazy_sum(const float* __restrict__ ys, const float* __restrict__ hs,
                                          size_t rs, int D, int t, int s0, int s1) {
  float a[kUnroll];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) a[u] = 0.f;
  int s = s0;
  for (; s + kUnroll <= s1; s += kUnroll) {
    float yv[kUnroll], hv[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      yv[u] = ys[(size_t)(s + u) * rs];
      hv[u] = hs[(size_t)(t - s - u) * D];
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) a[u] = fmaf(yv[u], hv[u], a[u]);
  }
  for (; s < s1; ++s) a[0] = fmaf(ys[(size_t)s * rs], hs[(size_t)(t - s) * D], a[0]);
#pragma unroll
  for (int w = kUnroll / 2; w >= 1; w /= 2)
#pragma unroll
    for (int u = 0; u < w; ++u) a[u] += a[u + w];
  return a[0];
}

// t <= kLazyCh: the whole step in one kernel.  Grid (column blocks, 1, layers).
__global__ __launch_bounds__(kBT) void k_lazy_fused(const float* __restrict__ y,
                                                   float* __restrict__ z, float* __restrict__ S,
                                                   const float* __restrict__ Hf, int m0, int L,
                                                   int BD, int D, int t) {
  const int c = (int)blockIdx.x * kBT + (int)threadIdx.x;
  if (c >= BD) return;
  const int m = m0 + (int)blockIdx.z;
  const int d = c % D;
  float* col = S + (size_t)m * L * BD + c;
  const float* hc = Hf + (size_t)m * L * D + d;
  const size_t e = (size_t)m * BD + c;
  const float yt = y[e];
  const float acc = lazy_sum(col, hc, (size_t)BD, D, t, 0, t);
  z[e] = fmaf(hc[0], yt, acc);
  col[(size_t)t * BD] = yt;
}

// Partial sums: chunk k = blockIdx.y covers s in [k kLazyCh, min((k+1) kLazyCh, t)).
__global__ __launch_bounds__(kBT) void k_lazy_partial(const float* __restrict__ S,
                                                     const float* __restrict__ Hf,
                                                     float* __restrict__ part, size_t pstride,
                                                     int m0, int L, int BD, int D, int t) {
  const int c = (int)blockIdx.x * kBT + (int)threadIdx.x;
  if (c >= BD) return;
  const int m = m0 + (int)blockIdx.z;
  const int d = c % D;
  const int s0 = (int)blockIdx.y * kLazyCh;
  const int s1 = s0 + kLazyCh < t ? s0 + kLazyCh : t;
  const float* col = S + (size_t)m * L * BD + c;
  const float* hc = Hf + (size_t)m * L * D + d;
  part[(size_t)blockIdx.y * pstride + (size_t)m * BD + c] =
      lazy_sum(col, hc, (size_t)BD, D, t, s0, s1);
}

// z_t = fmaf(h_0, y_t, sum of the nchunk partials in chunk order); y_t into the state.
__global__ __launch_bounds__(kBT) void k_lazy_reduce(const float* __restrict__ y,
                                                    float* __restrict__ z, float* __restrict__ S,
                                                    const float* __restrict__ Hf,
                                                    const float* __restrict__ part, size_t pstride,
                                                    int nchunk, int m0, int L, int BD, int D,
                                                    int t) {
  const int c = (int)blockIdx.x * kBT + (int)threadIdx.x;
  if (c >= BD) return;
  const int m = m0 + (int)blockIdx.z;
  const size_t e = (size_t)m * BD + c;
  const float yt = y[e];
  float acc = 0.f;
  for (int k = 0; k < nchunk; ++k) acc += part[(size_t)k * pstride + e];
  z[e] = fmaf(Hf[(size_t)m * L * D + c % D], yt, acc);
  S[(size_t)m * L * BD + (size_t)t * BD + c] = yt;
}

// Eager step t.  Grid (column blocks, row chunks (at least 1), layers): chunk
// k = blockIdx.y updates rows r in [t+1 + k kEagerCh, ...) below L; chunk 0
// also emits z_t from acc_t (a row no chunk writes).
__global__ __launch_bounds__(kBT) void k_eager_step(const float* __restrict__ y,
                                                   float* __restrict__ z, float* __restrict__ S,
                                                   const float* __restrict__ Hf, int m0, int L,
                                                   int BD, int D, int t) {
  const int c = (int)blockIdx.x * kBT + (int)threadIdx.x;
  if (c >= BD) return;
  const int m = m0 + (int)blockIdx.z;
  const int d = c % D;
  const size_t e = (size_t)m * BD + c;
  float* col = S + (size_t)m * L * BD + c;
  const float* hc = Hf + (size_t)m * L * D + d;
  const float yt = y[e];
  if (blockIdx.y == 0) z[e] = fmaf(hc[0], yt, col[(size_t)t * BD]);
  const int r0 = t + 1 + (int)blockIdx.y * kEagerCh;
  const int r1 = r0 + kEagerCh < L ? r0 + kEagerCh : L;
  int r = r0;
  for (; r + kUnroll <= r1; r += kUnroll) {
    float av[kUnroll], hv[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      av[u] = col[(size_t)(r + u) * BD];
      hv[u] = hc[(size_t)(r + u - t) * D];
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) col[(size_t)(r + u) * BD] = fmaf(yt, hv[u], av[u]);
  }
  for (; r < r1; ++r) col[(size_t)r * BD] = fmaf(yt, hc[(size_t)(r - t) * D], col[(size_t)r * BD]);
}

}  // namespace
}  // namespace lcsm

struct lcsm_base {
  lcsm::Shape s;
  int kind;  // LCSM_BASE_LAZY or LCSM_BASE_EAGER
  bool np;   // one launch per layer
  hipStream_t stream;
  bool owns_ws;
  char* ws;
  float* S;
  float* Hf;
  float* part;
  size_t pstride;  // M*B*D floats per partial-sum chunk
  int t;
  bool faulted;
  char msg[256];
};

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

struct BaseLayout {
  size_t S, Hf, part, total;
};

int check(int kind, int M, int B, int D, int L) {
  if (kind & ~(LCSM_BASE_EAGER | LCSM_BASE_NP)) return LCSM_EINVAL;
  if (M < 1 || B < 1 || D < 1 || L < 1) return LCSM_EINVAL;
  if (M > 65535 || B > 65535) return LCSM_EINVAL;
  if ((long long)M * B * D >= (1LL << 31)) return LCSM_EINVAL;
  if (L > (1 << 19)) return LCSM_EINVAL;
  return LCSM_OK;
}

BaseLayout base_layout(int kind, int M, int B, int D, int L) {
  BaseLayout ly{};
  const size_t cols = (size_t)M * B * D;
  size_t off = 0;
  ly.S = off;
  off = align_up(off + sizeof(float) * cols * L);
  ly.Hf = off;
  off = align_up(off + sizeof(float) * (size_t)M * L * D);
  ly.part = off;
  if ((kind & LCSM_BASE_EAGER) == 0) {
    const size_t nchunk = ((size_t)L + lcsm::kLazyCh - 1) / lcsm::kLazyCh;
    off = align_up(off + sizeof(float) * cols * nchunk);
  }
  ly.total = off;
  return ly;
}

int base_fail(lcsm_base* c, int code, const char* what, hipError_t e) {
  if (e != hipSuccess) {
    snprintf(c->msg, sizeof(c->msg), "%s: %s", what, hipGetErrorString(e));
    c->faulted = true;
    return LCSM_EDEVICE;
  }
  snprintf(c->msg, sizeof(c->msg), "%s", what);
  return code;
}

hipError_t lazy_step(lcsm_base* c, const float* y, float* z, int m0, int nm) {
  using namespace lcsm;
  const Shape& s = c->s;
  const int t = c->t;
  const dim3 block(kBT);
  if (t <= kLazyCh) {
    hipLaunchKernelGGL(k_lazy_fused, dim3(col_blocks(s.BD), 1, nm), block, 0, c->stream, y, z, c->S,
                       c->Hf, m0, s.L, s.BD, s.D, t);
    return hipGetLastError();
  }
  const int nchunk = (t + kLazyCh - 1) / kLazyCh;
  hipLaunchKernelGGL(k_lazy_partial, dim3(col_blocks(s.BD), nchunk, nm), block, 0, c->stream, c->S,
                     c->Hf, c->part, c->pstride, m0, s.L, s.BD, s.D, t);
  hipLaunchKernelGGL(k_lazy_reduce, dim3(col_blocks(s.BD), 1, nm), block, 0, c->stream, y, z, c->S,
                     c->Hf, c->part, c->pstride, nchunk, m0, s.L, s.BD, s.D, t);
  return hipGetLastError();
}

hipError_t eager_step(lcsm_base* c, const float* y, float* z, int m0, int nm) {
  using namespace lcsm;
  const Shape& s = c->s;
  const int t = c->t;
  const int rows = s.L - 1 - t;
  const int nchunk = rows > 0 ? (rows + kEagerCh - 1) / kEagerCh : 1;
  hipLaunchKernelGGL(k_eager_step, dim3(col_blocks(s.BD), nchunk, nm), dim3(kBT), 0, c->stream, y,
                     z, c->S, c->Hf, m0, s.L, s.BD, s.D, t);
  return hipGetLastError();
}

}  // namespace

extern "C" {

int lcsm_base_workspace_bytes(int kind, int M, int B, int D, int L, size_t* bytes) {
  if (!bytes) return LCSM_EINVAL;
  const int r = check(kind, M, B, D, L);
  if (r) return r;
  *bytes = base_layout(kind, M, B, D, L).total;
  return LCSM_OK;
}

int lcsm_base_init(lcsm_base** out, int kind, const float* filters, int M, int B, int D, int L,
                   void* stream, void* workspace, size_t workspace_bytes) {
  if (!out) return LCSM_EINVAL;
  *out = nullptr;
  if (!filters) return LCSM_EINVAL;
  int r = check(kind, M, B, D, L);
  if (r) return r;
  const BaseLayout ly = base_layout(kind, M, B, D, L);
  if (workspace) {
    if (workspace_bytes < ly.total) return LCSM_ENOMEM;
    if (((uintptr_t)workspace) % kAlign) return LCSM_EINVAL;
  }
  lcsm_base* c = new (std::nothrow) lcsm_base();
  if (!c) return LCSM_ENOMEM;
  c->s = lcsm::Shape{M, B, D, L, B * D, L};
  c->kind = kind & LCSM_BASE_EAGER;
  c->np = (kind & LCSM_BASE_NP) != 0;
  c->stream = (hipStream_t)stream;
  if (workspace) {
    c->ws = (char*)workspace;
    c->owns_ws = false;
  } else {
    void* p = nullptr;
    if (hipMalloc(&p, ly.total) != hipSuccess) {
      (void)hipGetLastError();
      delete c;
      return LCSM_ENOMEM;
    }
    c->ws = (char*)p;
    c->owns_ws = true;
  }
  c->S = (float*)(c->ws + ly.S);
  c->Hf = (float*)(c->ws + ly.Hf);
  c->part = (float*)(c->ws + ly.part);
  c->pstride = (size_t)M * B * D;
  hipError_t e = lcsm::launch_transpose_filters(filters, c->Hf, c->s, c->stream);
  if (e == hipSuccess) e = lcsm::launch_zero(c->S, (size_t)M * L * B * D, c->stream);
  if (e != hipSuccess) {
    if (c->owns_ws) (void)hipFree(c->ws);
    delete c;
    return LCSM_EDEVICE;
  }
  c->t = 0;
  c->faulted = false;
  c->msg[0] = 0;
  *out = c;
  return LCSM_OK;
}

int lcsm_base_step(lcsm_base* c, const float* y, float* z) {
  if (!c) return LCSM_EINVAL;
  if (!y || !z) return base_fail(c, LCSM_EINVAL, "null input or output pointer", hipSuccess);
  if (c->faulted) return LCSM_ESTATE;
  if (c->t >= c->s.L) return LCSM_EDONE;
  const int M = c->s.M;
  hipError_t e = hipSuccess;
  // parallel: every layer in one launch (grid z); NP: one launch per layer
  const int nm = c->np ? 1 : M;
  for (int m0 = 0; e == hipSuccess && m0 < M; m0 += nm)
    e = c->kind == LCSM_BASE_EAGER ? eager_step(c, y, z, m0, nm) : lazy_step(c, y, z, m0, nm);
  if (e != hipSuccess) return base_fail(c, LCSM_EDEVICE, "baseline step launch", e);
  c->t += 1;
  return LCSM_OK;
}

int lcsm_base_reset(lcsm_base* c) {
  if (!c) return LCSM_EINVAL;
  const hipError_t e =
      lcsm::launch_zero(c->S, (size_t)c->s.M * c->s.L * c->s.BD, c->stream);
  if (e != hipSuccess) return base_fail(c, LCSM_EDEVICE, "reset", e);
  c->t = 0;
  c->faulted = false;
  c->msg[0] = 0;
  return LCSM_OK;
}

int lcsm_base_position(const lcsm_base* c, int* t) {
  if (!c || !t) return LCSM_EINVAL;
  *t = c->t;
  return LCSM_OK;
}

void lcsm_base_destroy(lcsm_base* c) {
  if (!c) return;
  (void)hipStreamSynchronize(c->stream);
  if (c->owns_ws) (void)hipFree(c->ws);
  delete c;
}

const char* lcsm_base_last_error(const lcsm_base* c) { return c ? c->msg : ""; }

}  // extern "C"
