/*
 * lcsm.h -- C ABI of the relaxed online long-convolution library for AMD
 * MI355X (gfx950).
 *
 * Operation (Oncescu et al., "Flash Inference", arXiv 2410.12982):
 * for every layer m < M, batch row b < B and channel d < D the library
 * evaluates, online, the causal long convolution of Eq. (onlineConv)
 *
 *     z^m_t[b,d] = sum_{s=0}^{t} y^m_s[b,d] * h[m,d,t-s],   t = 0..L-1
 *
 * (0-indexed), where y^m_t is handed in at step t and z^m_t is returned at
 * the same step, before y^m_{t+1} exists.  The work is tiled as in Alg. 1 /
 * Alg. 3: at step t the diagonal term y_t h_0 completes z_t (the "red
 * cell"); then, with i = t+1 and U the largest power of two dividing i, the
 * contribution of y[i-U, i) to z[i, i+U) (the "gray tile", Eq. taus, lags
 * 1..2U-1) is added for all layers in one batch.  Small tiles run as a direct
 * Toeplitz product, large ones as a 2U-point cyclic FFT with filter spectra
 * precomputed per tile size (Lemma 1, App. B).  When L is not a power of two
 * the destination window is clipped at L.
 *
 * Conventions
 *  - Every float pointer is a DEVICE pointer to fp32 data unless stated.
 *  - Every call that touches the device is asynchronous on the stream given
 *    to lcsm_init; buffers handed in must stay valid until the stream has
 *    passed the call.
 *  - Return values: LCSM_OK (0) or a negative LCSM_E* code.  No call throws
 *    or aborts.  Arguments are validated before any device work is queued.
 *  - A context is not thread safe; distinct contexts are independent.
 */
#ifndef LCSM_H
#define LCSM_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Error codes. */
#define LCSM_OK 0
#define LCSM_EINVAL (-1)  /* bad argument: null pointer, size < 1 or too large */
#define LCSM_ENOMEM (-2)  /* workspace too small, or the library's allocation failed */
#define LCSM_EDEVICE (-3) /* a HIP runtime call or kernel launch failed; the context is faulted */
#define LCSM_EDONE (-4)   /* all L positions have been emitted; nothing was queued */
#define LCSM_ESTATE (-5)  /* call out of sequence, or the context is faulted (see lcsm_reset) */

/* Tile kinds reported by lcsm_plan_tile. */
#define LCSM_TILE_NONE 0    /* no gray tile after this step (t = L-1) */
#define LCSM_TILE_DIRECT 1  /* direct Toeplitz kernel */
#define LCSM_TILE_FFT 2     /* 2U-point FFT, one LDS-resident pass */
#define LCSM_TILE_FFT_HBM 3 /* 2U-point FFT, multi-pass through HBM scratch */
#define LCSM_TILE_FFT_COL 4 /* 2U-point FFT on column chunks transposed into the scratch */
#define LCSM_TILE_FFT_CM 5  /* 2U-point FFT on the column-major mirror of the state (below) */

/* Tuning options.  A NULL pointer, or a field left at 0, selects the
 * library default. */
typedef struct lcsm_options {
  int direct_max_u;  /* tiles with U <= direct_max_u use the direct kernel (power of two, >= 1),
                        larger ones the FFT.  0: by shape -- direct up to U = 32, and at U = 64
                        while M*B*D < 2^14 */
  int lds_fft_max_n; /* FFT tiles with 2U <= lds_fft_max_n run in one LDS pass, larger ones in
                        three passes through scratch (power of two in [16, 8192]; default 8192) */
  int scratch_mib;   /* cap of the multi-pass FFT scratch in MiB (default 512); the scratch is
                        never smaller than one chunk of 16 complex columns */
  int half_state;    /* 1: keep only T state rows per layer instead of L, T the largest power
                        of two below L (App. C, "Storing Only Half of the Activations"); see
                        the note below.  0 (default): L rows */
  int col_fft_min_n; /* FFT tiles with col_fft_min_n <= 2U <= 32768 transpose chunks of their
                        columns into the scratch and transform each column as one contiguous
                        run (2U = 32768: as its even and odd bins, two 16384-point halves;
                        power of two >= 4; above 32768: never).  0: by shape -- from
                        2U = 2048 while M*B*D >= 2^14; with col_tile_form = 1 or
                        half_state from 2U = 8192 while M*B*D >= 2^14, from 4096 while
                        M*B*D >= 2^15 */
  int col_tile_form; /* how the tiles of the column-tile sizes reach contiguous columns.  0
                        (default): a column-major mirror of the state (LCSM_TILE_FFT_CM, see
                        below); 1: chunks transposed into the scratch and back for every
                        tile (LCSM_TILE_FFT_COL; no mirror memory).  With half_state the
                        transposed chunks are always used */
  int reserved[2];   /* must be zero */
} lcsm_options;

/* Column-major mirror (col_tile_form = 0).  With T0 the smallest tile side
 * of the column-tile sizes, the context keeps a second copy of every layer's
 * columns, pairs of real columns interleaved along time (C[m][pair][t]),
 * holding the inputs of the positions already passed and, for later
 * positions, the sums of the mirrored tiles.  After every position t with
 * i = t+1 a multiple of T0, the inputs of the last T0 positions are copied
 * in, the tile of i reads its U inputs and adds its U outputs as contiguous
 * runs of the mirror, and the mirrored sums of positions [i, i+T0) are
 * handed to the state before position i is emitted.  That costs 16 bytes
 * per column and position (8 more with tiles above 2U = 32768, whose outputs
 * still go to the state) instead of 20U bytes per column of every column
 * tile, and doubles the state memory. */

/* Half-state storage (lcsm_options.half_state = 1).  After position T-1 no
 * input y_s with s < T is read again, and before it no contribution lands at
 * a position >= T.  So the state keeps rows for positions [0, T) only, and
 * the gray tile of i = T (side T, the largest one) writes its outputs for
 * positions [T, L) over the rows of its own inputs, which it has already
 * read: workgroup by workgroup (one LDS pass) or chunk by chunk of columns
 * (multi-pass), each reading its columns' inputs before it stores any of
 * their outputs.  From then on state row r stands for position T + r.  Needs
 * no memory beyond the ordinary tile's; every output is bit-for-bit that of
 * the full-state context with col_tile_form = 1 (a zero's sign aside; the
 * column-tile sizes run on transposed chunks with half-state storage).  Requirements: the tile of
 * side T is an FFT tile (L > 2 * the direct limit), and a prefill prompt P
 * satisfies 2P <= T.  State memory: M*T*B*D floats instead of M*L*B*D. */

typedef struct lcsm_ctx lcsm_ctx;

/* Device bytes of the workspace a context of this shape needs: the state
 * M*L*B*D fp32 (M*T*B*D with half_state) -- the activations of Sec. 3.3,
 * one slot per position that holds the accumulator until the position's
 * input overwrites it --, filters M*L*D fp32, the filter spectra of the FFT
 * tile sizes (App. B's cached DFTs), FFT scratch and a few small buffers.
 * Host only: touches no device.
 * Errors: LCSM_EINVAL for sizes < 1, M > 16384, B > 65535, M*B*D >= 2^31, L > 2^19 or
 * bad options (half_state not 0 or 1, or 1 where the tile of side T would be
 * a direct tile). */
int lcsm_workspace_bytes(int M, int B, int D, int L, const lcsm_options* opt, size_t* bytes);

/* Create a context (Alg. 3's state: all activations zero, position t = 0).
 *   filters   device, [M][D][L] fp32: h[m,d,k] is the lag-k tap of layer m,
 *             channel d (the filter rho^m of the paper, one per channel).
 *             Copied (and re-laid out) during the call's stream work; the
 *             caller may free it once the stream has passed lcsm_init.
 *   stream    hipStream_t to queue all work on; NULL = the null stream.
 *   workspace device buffer of at least lcsm_workspace_bytes bytes, 256-byte
 *             aligned, owned by the caller and kept alive until
 *             lcsm_destroy; NULL makes the library allocate (and free) it.
 * Initialisation computes the filter spectra of every FFT tile size
 * (App. B).  Errors: LCSM_EINVAL, LCSM_ENOMEM, LCSM_EDEVICE; *out is NULL
 * on failure. */
int lcsm_init(lcsm_ctx** out, const float* filters, int M, int B, int D, int L, void* stream,
              void* workspace, size_t workspace_bytes, const lcsm_options* opt);

/* One position for all layers (Alg. 3 with the layers' inputs given):
 *   y_t  device [M][B][D]: the inputs y^m_t of every layer at position t.
 *   z_t  device [M][B][D]: receives z^m_t = fmaf(h[m,d,0], y^m_t, acc^m_t),
 *        where acc^m_t is the sum of all earlier contributions.
 * Then queues the gray tiles of i = t+1 for all layers and advances t.
 * y_t and z_t may not overlap each other or the workspace.
 * Errors: LCSM_EDONE once t = L; LCSM_ESTATE after a fault or between
 * lcsm_step_layer calls; LCSM_EINVAL for null pointers. */
int lcsm_step(lcsm_ctx* ctx, const float* y_t, float* z_t);

/* One position for all layers with the library's built-in elementwise chain
 * standing in for the blocks and the sampler of Alg. 3:
 *   y^0_0 = x^0_0,  y^0_t = 0.5 tanh(z^{M-1}_{t-1}) + x^0_t  (t >= 1),
 *   y^m_t = 0.5 tanh(z^{m-1}_t) + x^m_t                      (m >= 1).
 *   x_t  device [M][B][D] additive inputs;  z_t  device [M][B][D] outputs.
 * The rule is evaluated as y = (x + 1/2) - 1/(1 + e^{2z}), the same
 * function (absolute error below 3.3e-7 for |x| <= 3).  The last layer's
 * z_{t-1} is kept inside the context.  Same errors as lcsm_step. */
int lcsm_step_chain(lcsm_ctx* ctx, const float* x_t, float* z_t);

/* Red cell of one layer at the current position (the inner loop of Alg. 2 /
 * Alg. 3, for callers that run their own block between layers):
 *   y, z device [B][D].  Layers must be stepped in order 0..M-1, each once,
 *   and then lcsm_advance called.  Errors: LCSM_ESTATE when out of order. */
int lcsm_step_layer(lcsm_ctx* ctx, int layer, const float* y, float* z);

/* Gray tiles of i = t+1 for all layers, after lcsm_step_layer has run for
 * every layer at position t; advances t.  Errors: LCSM_ESTATE otherwise. */
int lcsm_advance(lcsm_ctx* ctx);

/* Views for callers that fuse the red cell into their own kernel (the
 * kernel that produces y_t, e.g. a block's epilogue), as the red line of
 * Alg. 1 / Alg. 3 allows: z^m_t = fmaf(h^m_0[d], y^m_t[b,d], acc^m_t[b,d]).
 *
 * lcsm_h0: *h0 = device pointer to the lag-0 taps, h^m_0[d] at
 *   (*h0)[m * *layer_stride + d] (the library's lag-major filter copy; valid
 *   until lcsm_destroy).  Host only.  Errors: LCSM_EINVAL for null pointers.
 *
 * lcsm_pending: *acc = device pointer to the accumulators of the current
 *   position t, acc^m_t[b,d] at (*acc)[m * *layer_stride + b*D + d]: the sum
 *   of all contributions of earlier positions (every one of them comes from
 *   a gray tile queued before step t, so the values are complete once the
 *   context's stream has passed the work queued so far).  The pointer is
 *   valid for position t only: the row moves with every step (and, with
 *   half_state, wraps at T).  Host only.  Errors: LCSM_EINVAL, LCSM_EDONE
 *   once t = L, LCSM_ESTATE after a fault.
 *
 * lcsm_commit: the caller has done the red cell of every layer at t in
 *   place, in stream order before this call: read acc^m_t from the pending
 *   row, computed z^m_t with the fmaf above, and written y^m_t over it (the
 *   slot of position t holds the input from then on, Sec. 3.3).  Queues the
 *   gray tiles of i = t+1 for all layers and advances t, as lcsm_advance.
 *   Errors: LCSM_EDONE once t = L, LCSM_ESTATE after a fault or between
 *   lcsm_step_layer calls, LCSM_EDEVICE. */
int lcsm_h0(const lcsm_ctx* ctx, const float** h0, size_t* layer_stride);
int lcsm_pending(lcsm_ctx* ctx, float** acc, size_t* layer_stride);
int lcsm_commit(lcsm_ctx* ctx);

/* Run n consecutive lcsm_step calls (n iterations of Alg. 3's loop over
 * positions): step k reads y + k*y_stride and writes z + k*z_stride (strides
 * in floats).  Equivalent to the loop of single steps, with one host call.
 * Errors as lcsm_step; stops at the first. */
int lcsm_run(lcsm_ctx* ctx, int n, const float* y, size_t y_stride, float* z, size_t z_stride);

/* n consecutive lcsm_step_chain calls (the workloads' closed loop, Alg. 3's
 * loop over positions with the built-in elementwise chain as its blocks and
 * sampler): step k reads x + k*x_stride and writes z + k*z_stride (device
 * pointers, strides in floats); the results equal those of the loop of
 * single steps bit for bit.  The chain couples the layers of one (b, d)
 * column only, and a direct tile of U <= 16 that starts inside an aligned
 * block of 32 positions reads and writes rows of that block only; so with
 * full-state storage, at most 30 layers and at most 8192 columns per layer
 * (B*D), every stretch of such positions runs as one launch that keeps each
 * column's block rows in registers, and only the larger tiles are launched
 * on their own.  Other shapes take one position at a time.  Errors as
 * lcsm_step_chain; stops at the first. */
int lcsm_run_chain(lcsm_ctx* ctx, int n, const float* x, size_t x_stride, float* z,
                   size_t z_stride);

/* lcsm_run for callers that cannot allocate device memory (code under HIP
 * graph capture, serving loops or harnesses that forbid hipMalloc): the same
 * n steps, arguments, results (to fp32 rounding) and errors as lcsm_run,
 * allocating nothing.  The FFT tiles' staging (column chunks and multi-pass
 * transforms), which lcsm_run takes from the context's workspace, comes from
 * a static device array of the library instead: 64 MiB per GPU, reserved
 * when the library is loaded and held until the process ends, enough for
 * one chunk of every tile a context can plan (contexts whose tiles would
 * need more are rejected with LCSM_EINVAL before any work is queued).  That
 * array is shared by every call on the same GPU and keeps the last call's
 * contents (the tiles write every element before reading it): calls that
 * overlap on one GPU -- two streams, two threads, two contexts -- race on it
 * and must be serialised by the caller.  Chunks may differ in size from
 * lcsm_run's, so results can differ from it in the last bits. */
int lcsm_run_noalloc(lcsm_ctx* ctx, int n, const float* y, size_t y_stride, float* z,
                     size_t z_stride);

/* ---- Replayed generations (App. B.2, "CPU Overhead: The silent performance
 * killer": the per-token launches of a generation are recorded once as HIP
 * graphs and replayed, so the host submits a few graph launches per
 * generation instead of one or two kernel launches per position).
 *
 * lcsm_graph_capture records lcsm_reset followed by n consecutive steps into
 * a chain of HIP graphs of at most seg_positions positions each (a step is
 * one or two kernel launches, a few hundred only at the largest tiles, so
 * every graph holds about 2 * seg_positions nodes, whatever n is).  Step k (k < n) reads
 *   in + (k mod in_ring) * in_stride      (device, [M][B][D] fp32)
 * and writes
 *   z + (k mod z_ring) * z_stride         (device, [M][B][D] fp32),
 * strides in floats; in_ring / z_ring = 0 mean n (no wrap-around).  flags = 0
 * records lcsm_step (in = y_t); flags = LCSM_GRAPH_CHAIN records the chained
 * steps as lcsm_run_chain runs them (in = x_t, the built-in tanh chain; the
 * same results as lcsm_step_chain).  seg_positions = 0
 * selects LCSM_GRAPH_DEFAULT_SEG; at most LCSM_GRAPH_MAX_SEG.
 * Nothing runs on the device during the call; the context's stream must be
 * a created stream (not the null stream) that is not capturing, and the
 * context must not be faulted or between lcsm_step_layer calls.  Afterwards
 * the context's position is n, as if the recorded work had been queued.
 * The graphs keep the pointers they were recorded with: in, z and the
 * context's workspace must stay valid while the graph object lives.
 * Errors: LCSM_EINVAL (null pointers, n outside [1, L], bad rings or
 * seg_positions, the null stream), LCSM_ESTATE, LCSM_EDEVICE (the capture or
 * the instantiation failed; nothing is left recorded, the context is
 * faulted until lcsm_reset). */
#define LCSM_GRAPH_CHAIN 1
#define LCSM_GRAPH_DEFAULT_SEG 8192
#define LCSM_GRAPH_MAX_SEG 16384
typedef struct lcsm_graph lcsm_graph;
int lcsm_graph_capture(lcsm_ctx* ctx, int flags, int n, const float* in, size_t in_stride,
                       int in_ring, float* z, size_t z_stride, int z_ring, int seg_positions,
                       lcsm_graph** out);

/* Queue every graph of the chain, in order, on the context's stream: the same
 * device work as lcsm_reset followed by the n recorded steps.  Leaves the
 * context at position n.  Errors: LCSM_EINVAL, LCSM_EDEVICE (the context is
 * then faulted). */
int lcsm_graph_launch(lcsm_graph* g);

/* Number of graphs in the chain (ceil(n / seg_positions)).  Host only. */
int lcsm_graph_segments(const lcsm_graph* g, int* nseg);

/* Release the graphs (after the stream has passed their last launch).  NULL
 * is ignored.  Must come before lcsm_destroy of its context. */
void lcsm_graph_destroy(lcsm_graph* g);

/* Prompt prefill (Sec. 2.3.1 "The Inference Problem"; the appendix on the
 * prefilling and autoregressive stages): with all P prompt inputs known, the
 * prompt's own outputs come from one transform instead of P online steps.
 *   y  device [P][M][B][D] prompt inputs y^m_t, position k at y + k*y_stride;
 *   z  device [P][M][B][D] receives z^m_t for t < P, at z + k*z_stride
 *      (strides in floats, as for lcsm_run).
 * P must be a power of two with 2P <= L (2P <= T with half_state), and the
 * context at position 0 (after
 * lcsm_init or lcsm_reset).  Afterwards the context is at position P in
 * exactly the state P calls of lcsm_step would leave (state rows < P hold the
 * prompt, rows >= P its contributions from the gray tile of i = P), so
 * lcsm_step / lcsm_run continue the generation.  When P is an FFT tile size
 * (above the direct crossover) the work is: copy the prompt into the state,
 * one 2P-point tile with the filter spectrum delayed by P rows (its outputs
 * are the causal convolution of the prompt), the same tile with the cached
 * spectrum; the spectra of tile size P are recomputed twice in place.  For a
 * direct tile size it runs the P ordinary steps.  Errors: LCSM_EINVAL (null
 * pointers, P not a power of two, 2P > L, or 2P > T with half_state),
 * LCSM_ESTATE (not at position 0, or faulted), LCSM_EDEVICE. */
int lcsm_prefill(lcsm_ctx* ctx, int P, const float* y, size_t y_stride, float* z, size_t z_stride);

/* Restart at position 0 with all activations zero (the initial state of
 * Alg. 1 / Alg. 3: every accumulator z_t = 0 before the first position);
 * keeps filters and spectra and clears a fault.  The state is cleared by a
 * fill kernel (no memset), so the call may be recorded into a graph.
 * Errors: LCSM_EDEVICE. */
int lcsm_reset(lcsm_ctx* ctx);

/* Current position t (the next step emits z_t).  Host only. */
int lcsm_position(const lcsm_ctx* ctx, int* t);

/* Host-only schedule query, no context needed: the gray tile queued after
 * step t of a length-L run.  *i = t+1, *U = largest power of two dividing i,
 * the tile reads y[i-U, i) and adds into z[i, i + *dst_len) with
 * *dst_len = min(U, L-i); *kind is the LCSM_TILE_* the library uses for it
 * with these options and shape.  For t = L-1 *kind = LCSM_TILE_NONE and the
 * other outputs are 0.  Errors: LCSM_EINVAL. */
int lcsm_plan_tile(int M, int B, int D, int L, const lcsm_options* opt, int t, int* i, int* U,
                   int* dst_len, int* kind);

/* The same schedule query for this context's shape and options (Alg. 3's
 * gray phase after step t; outputs as lcsm_plan_tile).  Host only.
 * Errors: LCSM_EINVAL for null pointers or t outside [0, L). */
int lcsm_tile(const lcsm_ctx* ctx, int t, int* i, int* U, int* dst_len, int* kind);

/* Release the context and, if the library allocated it, the workspace.
 * Waits for the context's stream.  NULL is ignored. */
void lcsm_destroy(lcsm_ctx* ctx);

/* Static description of an error code. */
const char* lcsm_strerror(int code);

/* Text of the last error recorded on this context ("" if none). */
const char* lcsm_last_error(const lcsm_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* LCSM_H */
