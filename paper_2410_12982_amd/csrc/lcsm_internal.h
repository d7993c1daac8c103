// Internal declarations shared by the library's HIP sources (not installed).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <vector>

#include "lcsm.h"

namespace lcsm {

// Host twiddle table of the FFT kernels: tw[n + m] = exp(-2 pi i m / n) for
// n = 1, 2, 4, ..., nmax and m < n (fp64 evaluation rounded to fp32).
std::vector<float2> twiddle_table(int nmax);

// Shape of one context.  State rows are indexed [m][t][b*D + d] (time-major:
// one position of one layer is a contiguous B*D slab), filters [m][k][d].
// A layer's state holds SL rows: L, or with half-state storage the largest
// power of two T below L.  The kernels take the state pointer of the
// current phase: the array itself while positions are below T, the array
// moved back by T rows after the swap (position p at row p - T), so they
// index rows by position in both phases.
struct Shape {
  int M, B, D, L;
  int BD;  // B * D
  int SL;  // state rows per layer
};

// Largest tile side handled by the fused red+direct kernels, and by the
// fused kernel of the built-in chain (one thread walks all layers there);
// the chain fuses its tiles up to kChainFusedMaxU only up to kChainFusedMaxM
// layers, and with more layers only up to kChainFusedManyU (the U = 1 tile,
// whose two operands per layer keep the all-layer walk bound by bandwidth;
// larger ones go to the all-layer tile launch, parallel over layers).
constexpr int kFusedMaxU = 64;
constexpr int kChainFusedMaxU = 32;
constexpr int kChainFusedMaxM = 1;
constexpr int kChainFusedManyU = 1;
// Output chunk of the generic direct tile kernel (U >= kDirectJ).
constexpr int kDirectJ = 16;

// [M][D][L] -> [M][L][D]
hipError_t launch_transpose_filters(const float* src, float* dst, const Shape& s, hipStream_t st);

// Red cells of all layers at position t; when 1 <= U <= kFusedMaxU the gray
// tile i = t+1 (side U, dst_len outputs) is fused in.  U == 0: red only.
hipError_t launch_step_fused(const float* y, float* z, float* S, const float* Hf, const Shape& s,
                             int t, int U, int dst_len, hipStream_t st);

// Same with the elementwise tanh chain as input rule (see lcsm_step_chain).
hipError_t launch_chain_fused(const float* x, float* z, float* S, const float* Hf, float* prev,
                              const Shape& s, int t, int U, int dst_len, hipStream_t st);

// The chained steps of positions [t0, t1) in one launch, for a stretch that
// lies inside one aligned block of kChainBlockW positions and whose gray
// tiles are direct with U <= kChainBlockW / 2 (the last position's tile only
// when tile_last).  Position t reads x slab (xs0 + t - t0) mod xring and
// writes z slab (zs0 + t - t0) mod zring.  Full-state contexts with at most
// kChainBlockMaxM layers; a workgroup takes kChainBlockCols columns of every
// layer, and the launch is used while the columns fill at most
// kChainBlockMaxGroups workgroups (one per compute unit: beyond that, the
// serial chain of each workgroup makes one launch per position faster).
constexpr int kChainBlockW = 32;
constexpr int kChainBlockMaxM = 30;
constexpr int kChainBlockWave0StoreM = 4;  // up to this many layers the chain wave stores z and y
constexpr int kChainBlockCols = 32;
constexpr int kChainBlockMaxGroups = 256;
hipError_t launch_chain_block(const float* x, size_t xst, int xring, int xs0, float* z,
                              size_t zst, int zring, int zs0, float* S, const float* Hf,
                              float* prev, const Shape& s, int t0, int t1, bool tile_last,
                              hipStream_t st);

// Red cell of one layer at position t.
hipError_t launch_red_layer(const float* y, float* z, float* S, const float* Hf, const Shape& s,
                            int layer, int t, hipStream_t st);

// Direct gray tile of all layers: y rows [i-U, i) -> z rows [i, i+dst_len).
hipError_t launch_direct_tile(float* S, const float* Hf, const Shape& s, int i, int U, int dst_len,
                              hipStream_t st);

// Fill n floats with zero (a kernel, so it is safe under graph capture).
hipError_t launch_zero(float* p, size_t n, hipStream_t st);

// Fill the first n floats of each of M layers (layer k at p + k*stride) with zero.
hipError_t launch_zero_rows(float* p, int M, size_t stride, size_t n, hipStream_t st);

// Prompt rows: copy y[t][m][:] (position stride y_stride floats) into state
// rows t < P of every layer.
hipError_t launch_rows_in(const float* y, size_t y_stride, float* S, const Shape& s, int P,
                          hipStream_t st);

// Copy state rows row0 + t (t < P) of every layer out to z[t][m][:]
// (position stride z_stride floats) and clear them.
hipError_t launch_rows_out_clear(float* S, const Shape& s, int row0, int P, float* z,
                                 size_t z_stride, hipStream_t st);

// ---- FFT tiles (lcsm_fft.hip)

// Largest and preferred column-DFT length of the multi-pass split
// (N = N1 * N2): when preferred-length rows would leave columns longer than
// kPreferredMidN1, the rows take their largest length kMaxRowN2 instead.
constexpr int kMaxMidN1 = 128;
constexpr int kPreferredMidN1 = 32;
// Preferred and largest row-FFT length of the multi-pass split.
constexpr int kPreferredRowN2 = 1024;
constexpr int kMaxRowN2 = 4096;
// Range of the single-pass limit lds_fft_max_n.
constexpr int kMinLdsFftN = 16;
constexpr int kMaxLdsFftN = 8192;

// Complex columns per multi-pass chunk for an N-point transform over
// total_cc complex columns when the scratch holds scratch_bytes (a multiple
// of 16, or 0 if the scratch cannot hold one chunk of 16).
int fft_multipass_chunk(int N, size_t scratch_bytes, int total_cc);

// Filter spectra of tile size U (N = 2U): Hout[m][k][d] = DFT_N(g[m,d,0:N))[k]
// / N for k = 0..U, with g the filter delayed by shift rows (g[r] = h[r -
// shift], zero for r < shift).  tw: twiddle table (see lcsm_fft_core.h).
// colmaj: stored channel-major instead, Hout[m][d][k] (the column tiles).
hipError_t launch_spectra(const float* Hf, float2* Hout, const float2* tw, const Shape& s, int U,
                          int shift, int lds_max_n, float2* scratch, size_t scratch_bytes,
                          hipStream_t st, bool colmaj = false);

// ---- FFT tiles on transposed column chunks (lcsm_fft_col.hip)

// Largest 2U of the column tiles.
constexpr int kMaxColFftN = 32768;
// Largest 2U transformed as one column in LDS; the next size runs as two
// halves of this size (even and odd bins).
constexpr int kMaxColFftN1 = 16384;

// From this many columns (M*B*D) a launch has workgroups enough for FFT tile
// panels of 8 complex columns at 2U = 128 and 256 (64-byte row runs), and
// with them the FFT tile of U = 64 is faster than the direct one.
constexpr long long kWidePanelMinCols = 1LL << 14;

// Columns per chunk of a column tile of side U with scratch_bytes of
// scratch (a multiple of 64, 0 if not even 64 columns fit).
int fft_col_chunk(int U, size_t scratch_bytes, long long total_cols);

// FFT gray tile of all layers on transposed column chunks: y rows [i-U, i)
// -> z rows [i, i+dst_len) (added), or stored over rows [i-U, i-U+dst_len)
// when in_place (the half-state swap).  Hc: channel-major spectra [m][d][k]
// of tile size U.  2U <= kMaxColFftN; above kMaxColFftN1 the tile needs
// scratch for 2U floats per column of a chunk (at least 64 columns).
hipError_t launch_fft_col_tile(float* S, const float2* Hc, const float2* tw, const Shape& s, int i,
                               int U, int dst_len, float2* scratch, size_t scratch_bytes,
                               hipStream_t st, bool in_place);

// FFT gray tile of all layers: y rows [i-U, i) -> z rows [i, i+dst_len),
// with the spectra H of tile size U.  Single LDS pass when 2U <= lds_max_n,
// else the chunked multi-pass transform through scratch.  in_place: the
// outputs are stored (not added) over the input rows [i-U, i-U+dst_len)
// instead -- the swap of half-state storage; every workgroup (single pass) or
// chunk of columns (multi-pass) reads all of its columns' inputs before it
// stores any of their outputs.
hipError_t launch_fft_tile(float* S, const float2* H, const float2* tw, const Shape& s, int i,
                           int U, int dst_len, int lds_max_n, float2* scratch,
                           size_t scratch_bytes, hipStream_t st, bool in_place = false);

// ---- FFT tiles on the column-major mirror (lcsm_fft_col.hip)

// Pairs of real columns per layer in the mirror C[m][p][t] (float2): batch
// rows 2q and 2q+1 of one channel when B is even (bpair, p = q*D + d), else
// neighbouring columns 2p and 2p+1 (PC = ceil(B*D/2), the last pair's second
// column absent when B*D is odd).
struct CmShape {
  int PC;     // pairs per layer
  int bpair;  // 1: batch pairs, 0: neighbouring columns
};

// C[m][p][t] = (S[m][t][a], S[m][t][b]) for positions t in [row0, row1).
hipError_t launch_cm_yin(const float* S, float2* C, const Shape& s, const CmShape& cm, int row0,
                         int row1, hipStream_t st);

// State rows t in [row0, row1) receive the mirrored accumulators C[m][p][t]:
// stored (the rows hold nothing else yet) or added.
hipError_t launch_cm_merge(const float2* C, float* S, const Shape& s, const CmShape& cm, int row0,
                           int row1, bool store, hipStream_t st);

// FFT gray tile of side U at position i on the mirror, all layers: inputs
// C[p][i-U, i), outputs j < dst_len into C[p][i+j] (stored when `store`, else
// added).  Hc: channel-major spectra of tile size U.  2U <= kMaxColFftN; 2U =
// kMaxColFftN needs scratch for U complex values per pair of a chunk.
hipError_t launch_cm_tile(float2* C, const float2* Hc, const float2* tw, const Shape& s,
                          const CmShape& cm, int i, int U, int dst_len, bool store,
                          float2* scratch, size_t scratch_bytes, hipStream_t st);

// ---- hooks for a caller that runs the red cells in its own kernels (the
// synthetic model, lcsm_synth.hip): between two steps of a context,
// begin_external_step reports the position t and the state of its phase;
// after the caller has done the red cells of every layer at t (state slot
// of position t: S + (m*SL + t)*BD + c, z = fmaf(Hf[m*L*D + d], y, slot),
// slot = y), end_external_step queues the gray tiles of i = t+1 for all
// layers and advances t.  Return codes as lcsm_step.
struct StepView {
  float* S;         // state pointer of the phase of position t
  const float* Hf;  // filters [M][L][D]
  Shape s;
  int t;
  hipStream_t stream;
};
int begin_external_step(lcsm_ctx* c, StepView* v);
int end_external_step(lcsm_ctx* c);

// Largest FFT length with the red cell fused into the tile kernel.
constexpr int kMaxRedFftN = 4096;

// Red cells of all layers at position t = i-1 (inputs yt, outputs zt, both
// [M][B][D]) fused with the single-pass FFT tile of side U (2U <= the LDS
// limit and <= kMaxRedFftN, dst_len >= 1).
hipError_t launch_red_fft_tile(const float* yt, float* zt, float* S, const float* Hf,
                               const float2* H, const float2* tw, const Shape& s, int i, int U,
                               int dst_len, hipStream_t st);

}  // namespace lcsm
