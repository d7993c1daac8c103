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
#include "lcsm_internal.h"

namespace lcsm {
namespace {

constexpr int kThreads = 256;
constexpr int kDdJ = 16;            // outputs per thread of the direct tile
constexpr int kDdDefaultDirectMaxU = 32;

// Red cells of all layers at position t (grid: column blocks x M).
__global__ __launch_bounds__(kThreads) void k_dd_red(const float* __restrict__ y,
                                                     const float* __restrict__ rho,
                                                     float* __restrict__ z, float* __restrict__ Y,
                                                     float* __restrict__ R, int L, int BD, int t) {
  const int c = (int)blockIdx.x * kThreads + (int)threadIdx.x;
  if (c >= BD) return;
  const int m = (int)blockIdx.y;
  const size_t e = (size_t)m * BD + c;
  float* ycol = Y + (size_t)m * L * BD + c;
  float* rcol = R + (size_t)m * L * BD + c;
  const float yt = y[e], rt = rho[e];
  const float acc = ycol[(size_t)t * BD];
  float zt;
  if (t == 0) {
    zt = fmaf(yt, rt, acc);
  } else {
    zt = fmaf(yt, rcol[0], fmaf(ycol[0], rt, acc));
  }
  z[e] = zt;
  ycol[(size_t)t * BD] = yt;
  rcol[(size_t)t * BD] = rt;
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
    for (int k = 0; k < 4; ++k)
      if (o->reserved[k] != 0) return LCSM_EINVAL;
    if (o->scratch_mib != 0 || o->half_state != 0) return LCSM_EINVAL;
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
  const int Umax = largest_u(L);
  if (Umax > r->direct_max_u && 2 * Umax > r->fft_max_n) return LCSM_EINVAL;
  return LCSM_OK;
}

size_t dd_bytes(int M, int B, int D, int L) {
  const size_t state = align_up(sizeof(float) * (size_t)M * L * B * D);
  return 2 * state;
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

// One tile of side U for all layers.
hipError_t dd_tile(lcsm_dd* c, bool square, int U, int lo, int d0, int dlen) {
  const dim3 grid((unsigned)((c->BD + lcsm::kThreads - 1) / lcsm::kThreads),
                  (unsigned)((dlen + lcsm::kDdJ - 1) / lcsm::kDdJ), (unsigned)c->M);
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
  *bytes = dd_bytes(M, B, D, L);
  return LCSM_OK;
}

int lcsm_dd_init(lcsm_dd** out, int M, int B, int D, int L, void* stream, void* workspace,
                 size_t workspace_bytes, const lcsm_options* opt) {
  if (!out) return LCSM_EINVAL;
  *out = nullptr;
  DdOptions o;
  int r = resolve(M, B, D, L, opt, &o);
  if (r) return r;
  const size_t need = dd_bytes(M, B, D, L);
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
  c->Y = (float*)c->ws;
  c->R = (float*)(c->ws + need / 2);
  if (lcsm::launch_zero((float*)c->ws, need / sizeof(float), c->stream) != hipSuccess) {
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
  hipLaunchKernelGGL(lcsm::k_dd_red,
                     dim3((unsigned)((c->BD + lcsm::kThreads - 1) / lcsm::kThreads), (unsigned)c->M),
                     dim3(lcsm::kThreads), 0, c->stream, y_t, rho_t, z_t, c->Y, c->R, c->L, c->BD,
                     t);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return dd_fail(c, LCSM_EDEVICE, "red-cell launch", e);
  // every power of two U dividing t+1 with 2U <= t+1
  const int i1 = t + 1;
  for (int U = 1; i1 % U == 0 && 2 * U <= i1; U *= 2) {
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
  const size_t n = dd_bytes(c->M, c->B, c->D, c->L) / sizeof(float);
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
