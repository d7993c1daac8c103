/*
 * lcsm_dd.h -- C ABI of the relaxed online convolution with data-dependent
 * filters (include lcsm.h for the error codes and lcsm_options).
 *
 * Operation (the appendix on data-dependent filters of Oncescu et al.,
 * "Flash Inference", arXiv 2410.12982, Alg. 5): for every layer m < M,
 * batch row b < B and channel d < D, the filter rho is itself revealed
 * online -- rho^m_t arrives at step t together with y^m_t -- and the
 * library returns, at the same step,
 *
 *     z^m_t[b,d] = sum_{j+k=t} y^m_j[b,d] * rho^m_k[b,d],   t = 0..L-1.
 *
 * Work per step t: the red cell z_t = acc_t + y_t rho_0 + y_0 rho_t (the
 * last term for t >= 1), then, for every power of two U dividing t+1 with
 * 2U <= t+1, the untruncated convolutions of two length-U blocks (van der
 * Hoeven's relaxed product, which the appendix follows):
 *   t+1 = 2U:   acc[2U, 4U-1)   += y[U,2U) (*) rho[U,2U);
 *   otherwise:  acc[t+1, t+2U) += y[U,2U) (*) rho[t-U+1, t+1)
 *                                 + rho[U,2U) (*) y[t-U+1, t+1);
 * outputs past L-1 are dropped.  Tiles of one U run for all layers in one
 * launch; small ones directly, large ones as 2U-point FFTs.
 *
 * Conventions as in lcsm.h: device fp32 pointers, asynchronous on the
 * context's stream, LCSM_* return codes, arguments validated before any
 * device work is queued, not thread safe.
 */
#ifndef LCSM_DD_H
#define LCSM_DD_H

#include <stddef.h>

#include "lcsm.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lcsm_dd lcsm_dd;

/* Device bytes of the workspace (the inputs y and rho of every position:
 * 2*M*L*B*D fp32, the outputs' accumulators sharing y's rows, plus the FFT
 * twiddle table).  opt: direct_max_u (largest U done directly, default 32) and
 * lds_fft_max_n (largest transform of the FFT tiles, power of two in
 * [16, 8192], default 8192) apply; scratch_mib, half_state and col_fft_min_n
 * must be 0.  A tile with 2U above lds_fft_max_n = 2V runs as (U/V)^2 pairs
 * of V-blocks whose 2V-point product spectra are summed per output block
 * (same sums, more transforms).  Host only.
 * Errors: LCSM_EINVAL for the shapes lcsm_workspace_bytes rejects or bad
 * options. */
int lcsm_dd_workspace_bytes(int M, int B, int D, int L, const lcsm_options* opt, size_t* bytes);

/* Create a context at position 0 (all activations zero).  workspace: device
 * buffer of at least lcsm_dd_workspace_bytes bytes, 256-byte aligned, owned
 * by the caller until lcsm_dd_destroy, or NULL to let the library allocate
 * it.  Errors: LCSM_EINVAL, LCSM_ENOMEM, LCSM_EDEVICE; *out is NULL on
 * failure. */
int lcsm_dd_init(lcsm_dd** out, int M, int B, int D, int L, void* stream, void* workspace,
                 size_t workspace_bytes, const lcsm_options* opt);

/* One position for all layers: y_t, rho_t device [M][B][D] (inputs), z_t
 * device [M][B][D] (receives z_t).  Then queues the tiles of step t and
 * advances t.  The three buffers may not overlap each other or the
 * workspace.  Errors: LCSM_EDONE once t = L, LCSM_ESTATE after a fault,
 * LCSM_EINVAL for null pointers, LCSM_EDEVICE. */
int lcsm_dd_step(lcsm_dd* ctx, const float* y_t, const float* rho_t, float* z_t);

/* Back to position 0 with all activations zero; clears a fault.
 * Errors: LCSM_EDEVICE. */
int lcsm_dd_reset(lcsm_dd* ctx);

/* Current position t (the next step emits z_t).  Host only. */
int lcsm_dd_position(const lcsm_dd* ctx, int* t);

/* Release the context (waits for its stream) and, if the library allocated
 * it, the workspace.  NULL is ignored. */
void lcsm_dd_destroy(lcsm_dd* ctx);

/* Text of the last error recorded on this context ("" if none). */
const char* lcsm_dd_last_error(const lcsm_dd* ctx);

#ifdef __cplusplus
}
#endif

#endif /* LCSM_DD_H */
