// C ABI of the relaxed online convolution library: context, workspace,
// argument checks and the per-step tile scheduler (Alg. 1 / Alg. 3).
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <new>
#include <vector>

#include "lcsm.h"
#include "lcsm_internal.h"

using lcsm::Shape;

namespace {

constexpr size_t kAlign = 256;
// Default tile-kind choice (the paper's per-shape "Hybrid" choice of tau, from
// MI355X measurements): direct tiles (fused with the red cell) up to U = 32,
// and at U = 64 below kWidePanelMinCols columns, where the FFT tile of
// 2U = 128 runs in narrow panels and the launch is bound by its latency.
constexpr int kAutoDirectMaxU = 32;
constexpr int kDefaultLdsFftMaxN = 8192;   // 2U <= 8192: one LDS pass
constexpr int kDefaultScratchMib = 512;    // multi-pass and column-tile FFT scratch cap
// FFT tiles from 2U = 2048 up (to 32768) run as column tiles when there are
// at least 2^14 columns (M*B*D): on the column-major mirror they read and
// write contiguous runs, where the row-panel tile of 2U = 2048 holds one
// workgroup per CU and 64-byte row runs (measured per smallest column size,
// 1M / 55K / 18K columns: 2048 465 / 127.0 / 423 ms per generation, 4096 475
// / 127.9 / 426, 1024 490 / 131.5 / 438).  With the transposed chunks
// (col_tile_form = 1) the two transposes per tile make the column tiles pay
// only from 2U = 8192, and 4096 from 2^15 columns.
constexpr int kDefaultColFftMinN = 2048;
constexpr int kTransposedColFftMinN = 8192;
constexpr long long kAutoColMinCols = 1LL << 14;
constexpr long long kAutoCol4096MinCols = 1LL << 15;
constexpr int kMaxL = 1 << 19;             // FFT lengths up to 2^19 are built
constexpr int kMaxLevels = 20;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

bool is_pow2(int v) { return v > 0 && (v & (v - 1)) == 0; }

int lowbit(int i) { return i & -i; }

struct Options {
  int direct_max_u;  // 0: the shape-dependent default
  int lds_fft_max_n;
  int scratch_mib;
  int half_state;
  int col_min_n;
  bool col_auto;  // col_min_n is the default: applies from kAutoColMinCols columns
  int col_form;   // 0: column-major mirror, 1: transposed column chunks
};

int resolve_options(const lcsm_options* o, Options* r) {
  r->direct_max_u = 0;
  r->lds_fft_max_n = kDefaultLdsFftMaxN;
  r->scratch_mib = kDefaultScratchMib;
  r->half_state = 0;
  r->col_min_n = kDefaultColFftMinN;
  r->col_auto = true;
  r->col_form = 0;
  if (!o) return LCSM_OK;
  for (int k = 0; k < 2; ++k)
    if (o->reserved[k] != 0) return LCSM_EINVAL;
  if (o->col_tile_form != 0 && o->col_tile_form != 1) return LCSM_EINVAL;
  r->col_form = o->col_tile_form;
  if (o->col_fft_min_n) {
    if (!is_pow2(o->col_fft_min_n) || o->col_fft_min_n < 4) return LCSM_EINVAL;
    r->col_min_n = o->col_fft_min_n;
    r->col_auto = false;
  }
  if (o->direct_max_u < 0 || o->lds_fft_max_n < 0 || o->scratch_mib < 0) return LCSM_EINVAL;
  if (o->half_state != 0 && o->half_state != 1) return LCSM_EINVAL;
  r->half_state = o->half_state;
  if (o->direct_max_u) {
    if (!is_pow2(o->direct_max_u)) return LCSM_EINVAL;
    r->direct_max_u = o->direct_max_u;
  }
  if (o->lds_fft_max_n) {
    if (!is_pow2(o->lds_fft_max_n) || o->lds_fft_max_n < lcsm::kMinLdsFftN ||
        o->lds_fft_max_n > lcsm::kMaxLdsFftN)
      return LCSM_EINVAL;
    r->lds_fft_max_n = o->lds_fft_max_n;
  }
  if (o->scratch_mib) r->scratch_mib = o->scratch_mib;
  return LCSM_OK;
}

int check_shape(int M, int B, int D, int L) {
  if (M < 1 || B < 1 || D < 1 || L < 1) return LCSM_EINVAL;
  // grid y/z extents of the step kernels (z = M times the tile's thread split, <= 4)
  if (M > 16384 || B > 65535) return LCSM_EINVAL;
  if ((long long)M * B * D >= (1LL << 31)) return LCSM_EINVAL;
  if (L > kMaxL) return LCSM_EINVAL;
  return LCSM_OK;
}

int tile_kind(const Options& o, const Shape& s, int U) {
  if (U <= 0) return LCSM_TILE_NONE;
  int dmax = o.direct_max_u;
  if (dmax == 0)
    dmax = ((long long)s.M * s.BD < lcsm::kWidePanelMinCols) ? 2 * kAutoDirectMaxU : kAutoDirectMaxU;
  if (U <= dmax) return LCSM_TILE_DIRECT;
  const long long cols = (long long)s.M * s.BD;
  const bool mirror = o.col_form == 0 && !o.half_state;
  int col_min = o.col_min_n;
  if (o.col_auto && !mirror) col_min = cols >= kAutoCol4096MinCols ? 4096 : kTransposedColFftMinN;
  if (2 * U >= col_min && 2 * U <= lcsm::kMaxColFftN && (!o.col_auto || cols >= kAutoColMinCols))
    return mirror ? LCSM_TILE_FFT_CM : LCSM_TILE_FFT_COL;
  return (2 * U <= o.lds_fft_max_n) ? LCSM_TILE_FFT : LCSM_TILE_FFT_HBM;
}

// Shape with its state rows per layer: L, or with half-state storage (App. C)
// T = the largest power of two below L, the side of the largest tile (i = T).
// Half-state needs that tile to be an FFT tile: only those can store their
// outputs over their own inputs (-1 otherwise).
int make_shape(int M, int B, int D, int L, const Options& o, Shape* out) {
  Shape s{M, B, D, L, B * D, L};
  if (o.half_state) {
    if (L < 2) return LCSM_EINVAL;
    int T = 1;
    while (2 * T < L) T *= 2;
    s.SL = T;
    if (tile_kind(o, s, T) == LCSM_TILE_DIRECT) return LCSM_EINVAL;
  }
  *out = s;
  return LCSM_OK;
}

// Offsets of the workspace sections, in bytes.
struct Layout {
  size_t S, Hf, prev, tw, scratch, scratch_bytes, total;
  size_t scratch_min;    // bytes of one chunk of the largest multi-pass or column tile
  size_t C;              // the column-major mirror (when cm_t0 > 0)
  lcsm::CmShape cm;
  int cm_t0;             // smallest mirrored tile side (0: no mirror)
  unsigned cm_mask;      // OR of the mirrored tile sides
  bool cm_store;         // every tile side >= cm_t0 is mirrored: merges store
  size_t H[kMaxLevels];  // spectra of tile size 2^q (FFT levels only)
  int nmax;              // largest FFT length, 0 if no tile uses the FFT
};

Layout layout_for(const Shape& s, const Options& o) {
  Layout ly{};
  size_t off = 0;
  ly.S = off;
  off = align_up(off + sizeof(float) * (size_t)s.M * s.SL * s.BD);
  ly.Hf = off;
  off = align_up(off + sizeof(float) * (size_t)s.M * s.L * s.D);
  ly.prev = off;
  off = align_up(off + sizeof(float) * (size_t)s.BD);
  bool multipass = false, colsplit = false;
  ly.cm_store = true;
  for (int q = 0; q < kMaxLevels && (1 << q) <= s.L - 1; ++q) {
    const int U = 1 << q;
    const int kind = tile_kind(o, s, U);
    if (kind == LCSM_TILE_DIRECT) continue;
    ly.nmax = 2 * U;
    // the mirrored tiles take the column tiles' scratch: prefill's delayed
    // tile runs as a column tile, and 2U = 32768 needs it for its odd half
    if (kind == LCSM_TILE_FFT_HBM || kind == LCSM_TILE_FFT_COL || kind == LCSM_TILE_FFT_CM)
      multipass = true;
    if ((kind == LCSM_TILE_FFT_COL || kind == LCSM_TILE_FFT_CM) && 2 * U > lcsm::kMaxColFftN1)
      colsplit = true;
    if (kind == LCSM_TILE_FFT_CM) {
      if (!ly.cm_t0) ly.cm_t0 = U;
      ly.cm_mask |= (unsigned)U;
    } else if (ly.cm_t0) {
      ly.cm_store = false;  // a larger tile writes the state itself: merges add
    }
    ly.H[q] = off;
    off = align_up(off + sizeof(float2) * (size_t)s.M * (U + 1) * s.D);
  }
  if (ly.cm_t0) {
    ly.cm.bpair = s.B % 2 == 0 ? 1 : 0;
    ly.cm.PC = ly.cm.bpair ? (s.B / 2) * s.D : (s.BD + 1) / 2;
    ly.C = off;
    off = align_up(off + sizeof(float2) * (size_t)s.M * ly.cm.PC * s.L);
  }
  if (ly.nmax) {
    ly.tw = off;
    off = align_up(off + sizeof(float2) * 2 * (size_t)ly.nmax);
  }
  if (multipass) {
    // one chunk: N complex values per complex column (column tiles: U
    // floats per real column, the same bytes; split column tiles 2U, so 64
    // real columns need 32 complex columns' worth)
    const size_t per_col = sizeof(float2) * (size_t)ly.nmax;
    const size_t cols = ((size_t)s.M * ((s.BD + 1) / 2) + 15) / 16 * 16;
    const size_t min_cols = colsplit ? 32 : 16;
    size_t want = (size_t)o.scratch_mib << 20;
    if (want > per_col * cols) want = per_col * cols;
    if (want < per_col * min_cols) want = per_col * min_cols;
    ly.scratch = off;
    ly.scratch_bytes = want;
    ly.scratch_min = per_col * min_cols;
    off = align_up(off + want);
  }
  ly.total = off;
  return ly;
}

}  // namespace

// Staging of the FFT tiles for lcsm_run_noalloc (column chunks and the
// multi-pass scratch), in place of the workspace's scratch section: one
// array per GPU, loaded with the library and held until the process ends.
// Host code uses only its device address, resolved per device by
// static_scratch_ptr.  64 MiB holds one chunk of every tile the library
// builds (16 complex columns of the longest, 2^19-point, multi-pass
// transform).
constexpr size_t kStaticScratchBytes = 64ull << 20;
static __device__ __align__(256) float2 scratch[kStaticScratchBytes / sizeof(float2)];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float2* g_scratch_ptr[kMaxDevices];  // device address of scratch per device, null until resolved

// Device address of the static scratch on the current device (which must be
// `device`), looked up once per device.
hipError_t static_scratch_ptr(int device, float2** out) {
  *out = nullptr;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[device] = static_cast<float2*>(p);
  }
  *out = g_scratch_ptr[device];
  return hipSuccess;
}

}  // namespace

namespace lcsm {

// Twiddle table tw[n + m] = exp(-2 pi i m / n) for n = 1, 2, 4, ..., nmax.
std::vector<float2> twiddle_table(int nmax) {
  std::vector<float2> t(2 * (size_t)nmax);
  t[0] = make_float2(0.f, 0.f);
  t[1] = make_float2(1.f, 0.f);
  for (int n = 2; n <= nmax; n *= 2)
    for (int m = 0; m < n; ++m) {
      const double a = 2.0 * M_PI * (double)m / (double)n;
      t[(size_t)n + m] = make_float2((float)cos(a), (float)-sin(a));
    }
  return t;
}

}  // namespace lcsm

struct lcsm_ctx {
  Shape s;
  Options opt;
  Layout ly;
  hipStream_t stream;
  int device;
  bool owns_ws;
  char* ws;
  size_t ws_bytes;
  float* S;
  float* Hf;
  float* prev;
  float2* tw;
  float2* scratch;
  float2* C;               // column-major mirror (ly.cm_t0 > 0)
  int mirrored;            // positions [0, mirrored) of the mirror hold inputs
  float2* static_scratch;  // this device's static scratch (lcsm_run_noalloc)
  int T;            // half-state swap position (the state's rows per layer), 0 without
  int t;            // next position to emit
  int layers_done;  // lcsm_step_layer progress at position t
  bool faulted;
  char msg[256];
};

namespace {

int fail(lcsm_ctx* c, int code, const char* what, hipError_t e) {
  if (e != hipSuccess) {
    snprintf(c->msg, sizeof(c->msg), "%s: %s", what, hipGetErrorString(e));
    c->faulted = true;
    return LCSM_EDEVICE;
  }
  snprintf(c->msg, sizeof(c->msg), "%s", what);
  return code;
}

// Spectra of tile size U, in the layout of the level's tile kernel
// (channel-major for the column tiles), of the filter delayed by shift rows.
hipError_t spectra(lcsm_ctx* c, int U, int shift) {
  const int q = __builtin_ctz((unsigned)U);
  return lcsm::launch_spectra(c->Hf, (float2*)(c->ws + c->ly.H[q]), c->tw, c->s, U, shift,
                              c->opt.lds_fft_max_n, c->scratch, c->ly.scratch_bytes, c->stream,
                              tile_kind(c->opt, c->s, U) >= LCSM_TILE_FFT_COL);
}

// FFT tile of side U for all layers with the level's kernel, on the
// time-major state (a mirrored size runs as a transposed column tile here:
// prefill's delayed-filter tile).
hipError_t fft_tile(lcsm_ctx* c, float* S, int i, int U, int dst_len, bool in_place) {
  const float2* H = (const float2*)(c->ws + c->ly.H[__builtin_ctz((unsigned)U)]);
  if (tile_kind(c->opt, c->s, U) >= LCSM_TILE_FFT_COL)
    return lcsm::launch_fft_col_tile(S, H, c->tw, c->s, i, U, dst_len, c->scratch,
                                     c->ly.scratch_bytes, c->stream, in_place);
  return lcsm::launch_fft_tile(S, H, c->tw, c->s, i, U, dst_len, c->opt.lds_fft_max_n, c->scratch,
                               c->ly.scratch_bytes, c->stream, in_place);
}

// State pointer of the phase that position p belongs to: the array itself
// before the half-state swap, the array moved back by T rows from position T
// on (position p at row p - T; every row touched then is >= T).  Integer
// arithmetic: the moved pointer lies outside the allocation.
float* state_base(const lcsm_ctx* c, int p) {
  if (!c->T || p < c->T) return c->S;
  return (float*)((uintptr_t)c->S - sizeof(float) * (size_t)c->T * c->s.BD);
}

// Gray tile of i = t+1 for all layers, when it was not fused into the red
// launch.  With half-state storage the tile of i = T (an FFT tile) stores
// its outputs for positions [T, L) over its inputs, rows [0, L - T).
//
// Column-major mirror: every i that is a multiple of T0 (the smallest
// mirrored side; U >= T0 there) first copies the inputs of the positions not
// yet mirrored into it, and after the tile hands the mirrored sums of
// positions [i, i+T0) to the state -- if any mirrored tile reached them,
// i.e. if i has a bit at a mirrored side.  A mirrored tile stores its
// outputs when no mirrored tile reached those positions before, i.e. when
// the bits of i above U are at no mirrored side, and adds them otherwise,
// so the mirror never needs clearing.
hipError_t launch_tile(lcsm_ctx* c, int i, int U, int dst_len) {
  const int kind = tile_kind(c->opt, c->s, U);
  const bool swap = c->T && i == c->T;
  if (kind == LCSM_TILE_DIRECT)
    return lcsm::launch_direct_tile(state_base(c, i), c->Hf, c->s, i, U, dst_len, c->stream);
  const int t0 = c->ly.cm_t0;
  const bool boundary = t0 && i % t0 == 0;
  hipError_t e = hipSuccess;
  if (boundary) {
    e = lcsm::launch_cm_yin(c->S, c->C, c->s, c->ly.cm, c->mirrored, i, c->stream);
    c->mirrored = i;
  }
  if (e != hipSuccess) return e;
  if (kind == LCSM_TILE_FFT_CM) {
    const float2* H = (const float2*)(c->ws + c->ly.H[__builtin_ctz((unsigned)U)]);
    const bool store = ((unsigned)i & ~(2u * (unsigned)U - 1u) & c->ly.cm_mask) == 0;
    e = lcsm::launch_cm_tile(c->C, H, c->tw, c->s, c->ly.cm, i, U, dst_len, store, c->scratch,
                             c->ly.scratch_bytes, c->stream);
  } else {
    e = fft_tile(c, swap ? c->S : state_base(c, i), i, U, dst_len, swap);
  }
  if (e == hipSuccess && boundary && ((unsigned)i & c->ly.cm_mask)) {
    const int r1 = i + t0 < c->s.L ? i + t0 : c->s.L;
    e = lcsm::launch_cm_merge(c->C, c->S, c->s, c->ly.cm, i, r1, c->ly.cm_store, c->stream);
  }
  return e;
}

// Clear the state for position 0.  With a mirror whose merges store, only
// rows [0, T0) are read before being written (a merge stores every later row
// before anything else touches it); otherwise all rows.
hipError_t clear_state(lcsm_ctx* c) {
  const size_t per_layer = (size_t)c->s.SL * c->s.BD;
  if (c->ly.cm_t0 && c->ly.cm_store)
    return lcsm::launch_zero_rows(c->S, c->s.M, per_layer, (size_t)c->ly.cm_t0 * c->s.BD,
                                  c->stream);
  return lcsm::launch_zero(c->S, (size_t)c->s.M * per_layer, c->stream);
}

// Filter spectra of every FFT tile size (the cached kernel DFTs).
hipError_t init_spectra(lcsm_ctx* c) {
  if (!c->ly.nmax) return hipSuccess;
  std::vector<float2> t = lcsm::twiddle_table(c->ly.nmax);
  hipError_t e = hipMemcpyAsync(c->tw, t.data(), t.size() * sizeof(float2), hipMemcpyHostToDevice,
                                c->stream);
  for (int q = 0; e == hipSuccess && q < kMaxLevels && (1 << q) <= c->s.L - 1; ++q) {
    const int U = 1 << q;
    if (tile_kind(c->opt, c->s, U) == LCSM_TILE_DIRECT) continue;
    e = spectra(c, U, 0);
  }
  // the host table must outlive the copy
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  return e;
}

int step_common(lcsm_ctx* c, const float* in, float* z, bool chain) {
  if (!c) return LCSM_EINVAL;
  if (!in || !z) return fail(c, LCSM_EINVAL, "null input or output pointer", hipSuccess);
  if (c->faulted) return LCSM_ESTATE;
  if (c->layers_done != 0) return fail(c, LCSM_ESTATE, "step during a per-layer position", hipSuccess);
  if (c->t >= c->s.L) return LCSM_EDONE;
  const int t = c->t, i = t + 1;
  const int U = (i < c->s.L) ? lowbit(i) : 0;
  const int dst_len = U ? (U < c->s.L - i ? U : c->s.L - i) : 0;
  const int kind = tile_kind(c->opt, c->s, U);
  // the half-state swap tile runs on its own, after the red cells
  const bool swap = c->T && i == c->T;
  // The chained step fuses its tiles for a single layer; with several, the
  // red cells run one thread per column through all layers, fusing only the
  // U = 1 tile, and the other tiles go to the ordinary all-layer tile launch
  // (parallel over layers).
  const bool fuse =
      kind == LCSM_TILE_DIRECT && !swap &&
      (chain ? (U <= lcsm::kChainFusedMaxU &&
                (c->s.M <= lcsm::kChainFusedMaxM || U <= lcsm::kChainFusedManyU))
             : U <= lcsm::kFusedMaxU);
  float* S = state_base(c, t);
  hipError_t e;
  if (!chain && !swap && kind == LCSM_TILE_FFT && dst_len > 0 && 2 * U <= lcsm::kMaxRedFftN) {
    // red cells fused into the single-pass FFT tile: one launch
    const float2* H = (const float2*)(c->ws + c->ly.H[__builtin_ctz((unsigned)U)]);
    e = lcsm::launch_red_fft_tile(in, z, S, c->Hf, H, c->tw, c->s, i, U, dst_len, c->stream);
    if (e != hipSuccess) return fail(c, LCSM_EDEVICE, "red-cell + FFT tile launch", e);
    c->t = t + 1;
    return LCSM_OK;
  }
  if (chain)
    e = lcsm::launch_chain_fused(in, z, S, c->Hf, c->prev, c->s, t, fuse ? U : 0, dst_len,
                                 c->stream);
  else
    e = lcsm::launch_step_fused(in, z, S, c->Hf, c->s, t, fuse ? U : 0, dst_len, c->stream);
  if (e != hipSuccess) return fail(c, LCSM_EDEVICE, "red-cell launch", e);
  if (!fuse && kind != LCSM_TILE_NONE) {
    e = launch_tile(c, i, U, dst_len);
    if (e != hipSuccess) return fail(c, LCSM_EDEVICE, "gray-tile launch", e);
  }
  c->t = t + 1;
  return LCSM_OK;
}

// n chained steps (as n calls of lcsm_step_chain, the same results bit for
// bit).  Where the shape allows (chain_block_fits), each stretch of
// positions inside one aligned block of kChainBlockW whose gray tiles are
// direct with U <= kChainBlockW / 2 runs as one launch; the position that
// ends a stretch has its FFT or larger tile launched as usual.  Otherwise
// one position at a time.  Step k reads x slab (xs0 + k) mod xring and
// writes z slab (zs0 + k) mod zring.
bool chain_block_fits(const lcsm_ctx* c) {
  const long long groups = ((long long)c->s.BD + lcsm::kChainBlockCols - 1) / lcsm::kChainBlockCols;
  return !c->T && c->s.M <= lcsm::kChainBlockMaxM && groups <= lcsm::kChainBlockMaxGroups;
}

int chain_run(lcsm_ctx* c, int n, const float* x, size_t xst, int xring, int xs0, float* z,
              size_t zst, int zring, int zs0) {
  if (!c) return LCSM_EINVAL;
  if (!x || !z) return fail(c, LCSM_EINVAL, "null input or output pointer", hipSuccess);
  if (c->faulted) return LCSM_ESTATE;
  if (c->layers_done != 0) return fail(c, LCSM_ESTATE, "step during a per-layer position", hipSuccess);
  const bool block = chain_block_fits(c);
  constexpr int W = lcsm::kChainBlockW;
  int k = 0;
  while (k < n) {
    if (c->t >= c->s.L) return LCSM_EDONE;
    if (!block) {
      const int r = step_common(c, x + (size_t)((xs0 + k) % xring) * xst,
                                z + (size_t)((zs0 + k) % zring) * zst, true);
      if (r) return r;
      ++k;
      continue;
    }
    // the stretch: positions t0 .. t1-1, ending at the block's end, the end
    // of the run, or the first position whose tile is not a small direct one
    const int t0 = c->t;
    const int bend = (t0 & ~(W - 1)) + W;
    int t1 = t0;
    bool tile_last = true;
    while (t1 < c->s.L && t1 < bend && t1 - t0 < n - k) {
      const int i = ++t1;  // the tile after position t1 - 1
      if (i >= c->s.L) break;
      const int U = lowbit(i);
      if (U > W / 2 || tile_kind(c->opt, c->s, U) != LCSM_TILE_DIRECT) {
        tile_last = false;
        break;
      }
    }
    hipError_t e = lcsm::launch_chain_block(x, xst, xring, (xs0 + k) % xring, z, zst, zring,
                                            (zs0 + k) % zring, c->S, c->Hf, c->prev, c->s, t0, t1,
                                            tile_last, c->stream);
    if (e != hipSuccess) return fail(c, LCSM_EDEVICE, "chained-steps launch", e);
    if (!tile_last) {
      const int i = t1, U = lowbit(i);
      const int dst_len = U < c->s.L - i ? U : c->s.L - i;
      e = launch_tile(c, i, U, dst_len);
      if (e != hipSuccess) return fail(c, LCSM_EDEVICE, "gray-tile launch", e);
    }
    k += t1 - t0;
    c->t = t1;
  }
  return LCSM_OK;
}

}  // namespace

namespace lcsm {

int begin_external_step(lcsm_ctx* c, StepView* v) {
  if (!c || !v) return LCSM_EINVAL;
  if (c->faulted) return LCSM_ESTATE;
  if (c->layers_done != 0) return fail(c, LCSM_ESTATE, "step during a per-layer position", hipSuccess);
  if (c->t >= c->s.L) return LCSM_EDONE;
  v->S = state_base(c, c->t);
  v->Hf = c->Hf;
  v->s = c->s;
  v->t = c->t;
  v->stream = c->stream;
  return LCSM_OK;
}

int end_external_step(lcsm_ctx* c) {
  if (!c) return LCSM_EINVAL;
  c->layers_done = c->s.M;
  return lcsm_advance(c);
}

}  // namespace lcsm

extern "C" {

int lcsm_workspace_bytes(int M, int B, int D, int L, const lcsm_options* opt, size_t* bytes) {
  if (!bytes) return LCSM_EINVAL;
  int r = check_shape(M, B, D, L);
  if (r) return r;
  Options o;
  if ((r = resolve_options(opt, &o))) return r;
  Shape s;
  if ((r = make_shape(M, B, D, L, o, &s))) return r;
  *bytes = layout_for(s, o).total;
  return LCSM_OK;
}

int lcsm_init(lcsm_ctx** out, const float* filters, int M, int B, int D, int L, void* stream,
              void* workspace, size_t workspace_bytes, const lcsm_options* opt) {
  if (!out) return LCSM_EINVAL;
  *out = nullptr;
  if (!filters) return LCSM_EINVAL;
  int r = check_shape(M, B, D, L);
  if (r) return r;
  Options o;
  if ((r = resolve_options(opt, &o))) return r;
  Shape s;
  if ((r = make_shape(M, B, D, L, o, &s))) return r;
  const Layout ly = layout_for(s, o);
  if (workspace) {
    if (workspace_bytes < ly.total) return LCSM_ENOMEM;
    if (((uintptr_t)workspace) % kAlign) return LCSM_EINVAL;
  }
  lcsm_ctx* c = new (std::nothrow) lcsm_ctx();
  if (!c) return LCSM_ENOMEM;
  c->s = s;
  c->opt = o;
  c->ly = ly;
  c->stream = (hipStream_t)stream;
  c->msg[0] = 0;
  if (hipGetDevice(&c->device) != hipSuccess ||
      static_scratch_ptr(c->device, &c->static_scratch) != hipSuccess) {
    (void)hipGetLastError();
    delete c;
    return LCSM_EDEVICE;
  }
  if (workspace) {
    c->ws = (char*)workspace;
    c->ws_bytes = workspace_bytes;
    c->owns_ws = false;
  } else {
    void* p = nullptr;
    if (hipMalloc(&p, ly.total) != hipSuccess) {
      (void)hipGetLastError();
      delete c;
      return LCSM_ENOMEM;
    }
    c->ws = (char*)p;
    c->ws_bytes = ly.total;
    c->owns_ws = true;
  }
  c->S = (float*)(c->ws + ly.S);
  c->Hf = (float*)(c->ws + ly.Hf);
  c->prev = (float*)(c->ws + ly.prev);
  c->tw = ly.nmax ? (float2*)(c->ws + ly.tw) : nullptr;
  c->scratch = ly.scratch_bytes ? (float2*)(c->ws + ly.scratch) : nullptr;
  c->C = ly.cm_t0 ? (float2*)(c->ws + ly.C) : nullptr;
  c->mirrored = 0;
  c->T = o.half_state ? s.SL : 0;
  hipError_t e = lcsm::launch_transpose_filters(filters, c->Hf, s, c->stream);
  if (e == hipSuccess) e = lcsm::launch_zero(c->S, (size_t)s.M * s.SL * s.BD, c->stream);
  if (e == hipSuccess) e = lcsm::launch_zero(c->prev, (size_t)s.BD, c->stream);
  if (e == hipSuccess) e = init_spectra(c);
  if (e != hipSuccess) {
    if (c->owns_ws) (void)hipFree(c->ws);
    delete c;
    return LCSM_EDEVICE;
  }
  c->t = 0;
  c->layers_done = 0;
  c->faulted = false;
  *out = c;
  return LCSM_OK;
}

int lcsm_step(lcsm_ctx* ctx, const float* y_t, float* z_t) {
  return step_common(ctx, y_t, z_t, false);
}

int lcsm_step_chain(lcsm_ctx* ctx, const float* x_t, float* z_t) {
  return step_common(ctx, x_t, z_t, true);
}

int lcsm_step_layer(lcsm_ctx* c, int layer, const float* y, float* z) {
  if (!c) return LCSM_EINVAL;
  if (!y || !z) return fail(c, LCSM_EINVAL, "null input or output pointer", hipSuccess);
  if (c->faulted) return LCSM_ESTATE;
  if (c->t >= c->s.L) return LCSM_EDONE;
  if (layer != c->layers_done)
    return fail(c, LCSM_ESTATE, "layers must be stepped in order 0..M-1", hipSuccess);
  hipError_t e =
      lcsm::launch_red_layer(y, z, state_base(c, c->t), c->Hf, c->s, layer, c->t, c->stream);
  if (e != hipSuccess) return fail(c, LCSM_EDEVICE, "red-cell launch", e);
  c->layers_done = layer + 1;
  return LCSM_OK;
}

int lcsm_advance(lcsm_ctx* c) {
  if (!c) return LCSM_EINVAL;
  if (c->faulted) return LCSM_ESTATE;
  if (c->t >= c->s.L) return LCSM_EDONE;
  if (c->layers_done != c->s.M)
    return fail(c, LCSM_ESTATE, "lcsm_advance before every layer was stepped", hipSuccess);
  const int i = c->t + 1;
  if (i < c->s.L) {
    const int U = lowbit(i);
    const int dst_len = U < c->s.L - i ? U : c->s.L - i;
    hipError_t e = launch_tile(c, i, U, dst_len);
    if (e != hipSuccess) return fail(c, LCSM_EDEVICE, "gray-tile launch", e);
  }
  c->layers_done = 0;
  c->t = i;
  return LCSM_OK;
}

int lcsm_run(lcsm_ctx* c, int n, const float* y, size_t y_stride, float* z, size_t z_stride) {
  if (!c) return LCSM_EINVAL;
  if (n < 0) return fail(c, LCSM_EINVAL, "negative step count", hipSuccess);
  for (int k = 0; k < n; ++k) {
    const int r = step_common(c, y + (size_t)k * y_stride, z + (size_t)k * z_stride, false);
    if (r) return r;
  }
  return LCSM_OK;
}

int lcsm_run_chain(lcsm_ctx* c, int n, const float* x, size_t x_stride, float* z, size_t z_stride) {
  if (!c) return LCSM_EINVAL;
  if (n < 0) return fail(c, LCSM_EINVAL, "negative step count", hipSuccess);
  if (n == 0) return LCSM_OK;
  return chain_run(c, n, x, x_stride, n, 0, z, z_stride, n, 0);
}

int lcsm_run_noalloc(lcsm_ctx* c, int n, const float* y, size_t y_stride, float* z,
                     size_t z_stride) {
  if (!c) return LCSM_EINVAL;
  if (n < 0) return fail(c, LCSM_EINVAL, "negative step count", hipSuccess);
  if (c->ly.scratch_min > kStaticScratchBytes)
    return fail(c, LCSM_EINVAL, "one chunk of the FFT tiles exceeds the 64 MiB static scratch",
                hipSuccess);
  if (!c->static_scratch) return fail(c, LCSM_EDEVICE, "static scratch unavailable", hipSuccess);
  // the same steps, with the FFT tiles staged in the static scratch
  float2* const ws_scratch = c->scratch;
  const size_t ws_bytes = c->ly.scratch_bytes;
  if (ws_bytes) {
    c->scratch = c->static_scratch;
    c->ly.scratch_bytes = kStaticScratchBytes;
  }
  int r = LCSM_OK;
  for (int k = 0; r == LCSM_OK && k < n; ++k)
    r = step_common(c, y + (size_t)k * y_stride, z + (size_t)k * z_stride, false);
  c->scratch = ws_scratch;
  c->ly.scratch_bytes = ws_bytes;
  return r;
}

}  // extern "C"

// A recorded generation: lcsm_reset plus n steps, split into graphs of at
// most seg positions so that no graph's node count grows with n.  A step is
// one or two kernel launches, a few hundred only at the rare largest tiles,
// so a graph holds about 2 seg nodes (at most 16384 positions: about 33k
// nodes).  Graphs of about 131k and 1.08M nodes crashed the process while
// they were recorded or instantiated; graphs of about 33k nodes are known
// good.
struct lcsm_graph {
  lcsm_ctx* ctx;
  int n;
  int mirrored;  // the context's mirrored positions after the recorded steps
  std::vector<hipGraph_t> graphs;
  std::vector<hipGraphExec_t> execs;
};

namespace {

void release_graphs(lcsm_graph* g) {
  for (hipGraphExec_t e : g->execs) (void)hipGraphExecDestroy(e);
  for (hipGraph_t gr : g->graphs) (void)hipGraphDestroy(gr);
  g->execs.clear();
  g->graphs.clear();
}

}  // namespace

extern "C" {

int lcsm_graph_capture(lcsm_ctx* c, int flags, int n, const float* in, size_t in_stride,
                       int in_ring, float* z, size_t z_stride, int z_ring, int seg,
                       lcsm_graph** out) {
  if (!out) return LCSM_EINVAL;
  *out = nullptr;
  if (!c) return LCSM_EINVAL;
  if (!in || !z) return fail(c, LCSM_EINVAL, "null input or output pointer", hipSuccess);
  if (flags != 0 && flags != LCSM_GRAPH_CHAIN)
    return fail(c, LCSM_EINVAL, "unknown graph flags", hipSuccess);
  if (n < 1 || n > c->s.L) return fail(c, LCSM_EINVAL, "position count outside [1, L]", hipSuccess);
  if (in_ring < 0 || z_ring < 0) return fail(c, LCSM_EINVAL, "negative ring length", hipSuccess);
  if (seg == 0) seg = LCSM_GRAPH_DEFAULT_SEG;
  if (seg < 1 || seg > LCSM_GRAPH_MAX_SEG)
    return fail(c, LCSM_EINVAL, "positions per graph outside [1, LCSM_GRAPH_MAX_SEG]", hipSuccess);
  if (!c->stream) return fail(c, LCSM_EINVAL, "graphs need a created stream, not the null stream", hipSuccess);
  if (c->faulted) return LCSM_ESTATE;
  if (c->layers_done != 0)
    return fail(c, LCSM_ESTATE, "capture during a per-layer position", hipSuccess);
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  hipError_t e = hipStreamIsCapturing(c->stream, &cs);
  if (e != hipSuccess) return fail(c, LCSM_EDEVICE, "stream capture status", e);
  if (cs != hipStreamCaptureStatusNone)
    return fail(c, LCSM_ESTATE, "the stream is already capturing", hipSuccess);
  const int ir = in_ring ? in_ring : n, zr = z_ring ? z_ring : n;
  const bool chain = flags == LCSM_GRAPH_CHAIN;
  lcsm_graph* g = new (std::nothrow) lcsm_graph();
  if (!g) return LCSM_ENOMEM;
  g->ctx = c;
  g->n = n;
  for (int p0 = 0; p0 < n; p0 += seg) {
    const int p1 = n - p0 < seg ? n : p0 + seg;
    e = hipStreamBeginCapture(c->stream, hipStreamCaptureModeThreadLocal);
    if (e != hipSuccess) break;
    int r = LCSM_OK;
    if (p0 == 0) r = lcsm_reset(c);
    if (chain) {
      if (r == LCSM_OK) r = chain_run(c, p1 - p0, in, in_stride, ir, p0 % ir, z, z_stride, zr, p0 % zr);
    } else {
      for (int t = p0; r == LCSM_OK && t < p1; ++t)
        r = step_common(c, in + (size_t)(t % ir) * in_stride, z + (size_t)(t % zr) * z_stride, false);
    }
    hipGraph_t gr = nullptr;
    e = hipStreamEndCapture(c->stream, &gr);
    if (gr) g->graphs.push_back(gr);
    if (r != LCSM_OK && e == hipSuccess) e = hipErrorLaunchFailure;
    if (e != hipSuccess) break;
    hipGraphExec_t ex = nullptr;
    e = hipGraphInstantiate(&ex, gr, nullptr, nullptr, 0);
    if (e != hipSuccess) break;
    g->execs.push_back(ex);
  }
  if (e != hipSuccess) {
    release_graphs(g);
    delete g;
    (void)hipGetLastError();
    return fail(c, LCSM_EDEVICE, "graph capture", e);
  }
  g->mirrored = c->mirrored;
  *out = g;
  return LCSM_OK;
}

int lcsm_graph_launch(lcsm_graph* g) {
  if (!g || !g->ctx) return LCSM_EINVAL;
  lcsm_ctx* c = g->ctx;
  for (hipGraphExec_t ex : g->execs) {
    const hipError_t e = hipGraphLaunch(ex, c->stream);
    if (e != hipSuccess) return fail(c, LCSM_EDEVICE, "graph launch", e);
  }
  // the host-side bookkeeping of the recorded steps' end (the graphs begin
  // with a reset, so nothing before the launch carries over)
  c->t = g->n;
  c->mirrored = g->mirrored;
  c->layers_done = 0;
  c->faulted = false;
  return LCSM_OK;
}

int lcsm_graph_segments(const lcsm_graph* g, int* nseg) {
  if (!g || !nseg) return LCSM_EINVAL;
  *nseg = (int)g->execs.size();
  return LCSM_OK;
}

void lcsm_graph_destroy(lcsm_graph* g) {
  if (!g) return;
  release_graphs(g);
  delete g;
}

int lcsm_prefill(lcsm_ctx* c, int P, const float* y, size_t y_stride, float* z, size_t z_stride) {
  if (!c) return LCSM_EINVAL;
  if (!y || !z) return fail(c, LCSM_EINVAL, "null input or output pointer", hipSuccess);
  if (c->faulted) return LCSM_ESTATE;
  if (c->t != 0 || c->layers_done != 0)
    return fail(c, LCSM_ESTATE, "prefill only at position 0 (after init or reset)", hipSuccess);
  if (!is_pow2(P) || 2 * P > c->s.L)
    return fail(c, LCSM_EINVAL, "prompt length must be a power of two with 2P <= L", hipSuccess);
  // with half-state storage the prompt's outputs need state rows [P, 2P)
  if (2 * P > c->s.SL)
    return fail(c, LCSM_EINVAL, "half-state storage: the prompt needs 2P <= T", hipSuccess);
  const Shape& s = c->s;
  // a prompt of a direct tile size: P ordinary steps
  if (tile_kind(c->opt, s, P) == LCSM_TILE_DIRECT) return lcsm_run(c, P, y, y_stride, z, z_stride);
  // P is an FFT tile size, so its cached spectra and the twiddles for 2P exist
  // the prompt into state rows [0, P)
  hipError_t e = lcsm::launch_rows_in(y, y_stride, c->S, s, P, c->stream);
  // rows [P, 2P) are clear after a reset unless a mirror's merges store (then
  // only rows below T0 are)
  if (e == hipSuccess && c->ly.cm_t0 && c->ly.cm_store && 2 * P > c->ly.cm_t0)
    e = lcsm::launch_zero_rows(c->S + (size_t)P * s.BD, s.M, (size_t)s.SL * s.BD,
                               (size_t)P * s.BD, c->stream);
  // the tile i = P with the filter delayed by P rows puts, in rows [P, 2P),
  // sum_{k<P} y[k] h[j - k] = z_j for j < P: the prompt's own outputs
  if (e == hipSuccess) e = spectra(c, P, P);
  if (e == hipSuccess) e = fft_tile(c, c->S, P, P, P, false);
  if (e == hipSuccess) e = lcsm::launch_rows_out_clear(c->S, s, P, P, z, z_stride, c->stream);
  // the tile spectra back, then the gray tile of i = P that P steps would end with
  if (e == hipSuccess) e = spectra(c, P, 0);
  if (e == hipSuccess) e = launch_tile(c, P, P, P);
  if (e != hipSuccess) return fail(c, LCSM_EDEVICE, "prefill", e);
  c->t = P;
  return LCSM_OK;
}

int lcsm_reset(lcsm_ctx* c) {
  if (!c) return LCSM_EINVAL;
  hipError_t e = clear_state(c);
  if (e == hipSuccess) e = lcsm::launch_zero(c->prev, (size_t)c->s.BD, c->stream);
  if (e != hipSuccess) return fail(c, LCSM_EDEVICE, "reset", e);
  c->t = 0;
  c->mirrored = 0;
  c->layers_done = 0;
  c->faulted = false;
  c->msg[0] = 0;
  return LCSM_OK;
}

int lcsm_position(const lcsm_ctx* c, int* t) {
  if (!c || !t) return LCSM_EINVAL;
  *t = c->t;
  return LCSM_OK;
}

int lcsm_plan_tile(int M, int B, int D, int L, const lcsm_options* opt, int t, int* i, int* U,
                   int* dst_len, int* kind) {
  if (!i || !U || !dst_len || !kind) return LCSM_EINVAL;
  int r = check_shape(M, B, D, L);
  if (r) return r;
  Options o;
  if ((r = resolve_options(opt, &o))) return r;
  if (t < 0 || t >= L) return LCSM_EINVAL;
  const int ii = t + 1;
  if (ii >= L) {
    *i = *U = *dst_len = 0;
    *kind = LCSM_TILE_NONE;
    return LCSM_OK;
  }
  const int u = lowbit(ii);
  *i = ii;
  *U = u;
  *dst_len = u < L - ii ? u : L - ii;
  Shape s;
  if ((r = make_shape(M, B, D, L, o, &s))) return r;
  *kind = tile_kind(o, s, u);
  return LCSM_OK;
}

int lcsm_tile(const lcsm_ctx* c, int t, int* i, int* U, int* dst_len, int* kind) {
  if (!c || !i || !U || !dst_len || !kind) return LCSM_EINVAL;
  if (t < 0 || t >= c->s.L) return LCSM_EINVAL;
  const int ii = t + 1;
  if (ii >= c->s.L) {
    *i = *U = *dst_len = 0;
    *kind = LCSM_TILE_NONE;
    return LCSM_OK;
  }
  const int u = lowbit(ii);
  *i = ii;
  *U = u;
  *dst_len = u < c->s.L - ii ? u : c->s.L - ii;
  *kind = tile_kind(c->opt, c->s, u);
  return LCSM_OK;
}

int lcsm_h0(const lcsm_ctx* c, const float** h0, size_t* layer_stride) {
  if (!c || !h0 || !layer_stride) return LCSM_EINVAL;
  *h0 = c->Hf;
  *layer_stride = (size_t)c->s.L * c->s.D;
  return LCSM_OK;
}

int lcsm_pending(lcsm_ctx* c, float** acc, size_t* layer_stride) {
  if (!c || !acc || !layer_stride) return LCSM_EINVAL;
  if (c->faulted) return LCSM_ESTATE;
  if (c->t >= c->s.L) return LCSM_EDONE;
  const int row = (c->T && c->t >= c->T) ? c->t - c->T : c->t;  // half-state: rows wrap at T
  *acc = c->S + (size_t)row * c->s.BD;
  *layer_stride = (size_t)c->s.SL * c->s.BD;
  return LCSM_OK;
}

int lcsm_commit(lcsm_ctx* c) {
  if (!c) return LCSM_EINVAL;
  if (c->faulted) return LCSM_ESTATE;
  if (c->t >= c->s.L) return LCSM_EDONE;
  if (c->layers_done != 0)
    return fail(c, LCSM_ESTATE, "lcsm_commit during a per-layer position", hipSuccess);
  c->layers_done = c->s.M;
  return lcsm_advance(c);
}

void lcsm_destroy(lcsm_ctx* c) {
  if (!c) return;
  (void)hipStreamSynchronize(c->stream);
  if (c->owns_ws) (void)hipFree(c->ws);
  delete c;
}

const char* lcsm_strerror(int code) {
  switch (code) {
    case LCSM_OK:
      return "ok";
    case LCSM_EINVAL:
      return "invalid argument";
    case LCSM_ENOMEM:
      return "workspace too small or allocation failed";
    case LCSM_EDEVICE:
      return "HIP runtime or kernel launch error";
    case LCSM_EDONE:
      return "all positions already emitted";
    case LCSM_ESTATE:
      return "call out of sequence or context faulted";
    default:
      return "unknown error code";
  }
}

const char* lcsm_last_error(const lcsm_ctx* c) { return c ? c->msg : ""; }

}  // extern "C"
