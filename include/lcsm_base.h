/*
 * lcsm_base.h -- C ABI of the lazy and eager online convolutions, the
 * baselines the relaxed tiling is measured against (Oncescu et al., "Flash
 * Inference", arXiv 2410.12982, Sec. 3.1.1 "Relaxed Polynomial
 * Interpolation" and Sec. 5, whose speed-ups are stated over the lazy
 * approach parallelised across layers).
 *
 * Both compute, for every layer m < M, batch row b < B, channel d < D and
 * position t (0-indexed), the same z^m_t[b,d] = sum_{s<=t} y^m_s[b,d] *
 * h[m,d,t-s] as lcsm_step (Eq. onlineConv), with y_t handed in at step t:
 *
 *  - LAZY:  at step t, z_t is computed from the formula: a sum over the t+1
 *    stored inputs y_0 .. y_t (O(t) work per position, the contributions
 *    grouped in thin horizontal strips);
 *  - EAGER: at step t, z_t = acc_t + h_0 y_t is emitted and y_t's
 *    contributions y_t h_k are added at once to every later accumulator
 *    acc_{t+k}, k = 1 .. L-1-t (O(L-t) work per position, vertical strips).
 *
 * With the LCSM_BASE_NP flag every layer is a launch of its own (the
 * variants the paper calls non-parallel, *_NP); without it one launch covers
 * all M layers (the paper's parallel Lazy / Eager, Sec. 3.2).
 *
 * Sums are taken in a fixed order (no atomics): results are deterministic.
 * Conventions as in lcsm.h: device pointers to fp32 data, every call that
 * touches the device asynchronous on the context's stream, negative LCSM_E*
 * codes on error, arguments validated before any device work.
 */
#ifndef LCSM_BASE_H
#define LCSM_BASE_H

#include <stddef.h>

#include "lcsm.h"

#ifdef __cplusplus
extern "C" {
#endif

#define LCSM_BASE_LAZY 0
#define LCSM_BASE_EAGER 1
#define LCSM_BASE_NP 2 /* flag: one launch per layer */

typedef struct lcsm_base lcsm_base;

/* Device bytes of the workspace of a baseline context (kind = LCSM_BASE_LAZY
 * or LCSM_BASE_EAGER, optionally | LCSM_BASE_NP): the state M*L*B*D fp32
 * (LAZY: the inputs y_s, EAGER: the accumulators acc_t), the filters
 * M*L*D fp32 and, for LAZY, the partial sums of the split reduction
 * (ceil(L/256) * M*B*D fp32).  Host only.  Errors: LCSM_EINVAL for a bad
 * kind or the shapes lcsm_workspace_bytes rejects. */
int lcsm_base_workspace_bytes(int kind, int M, int B, int D, int L, size_t* bytes);

/* Create a baseline context at position 0 (state zero).  filters: device
 * [M][D][L] fp32, copied during the call's stream work.  stream: hipStream_t
 * (NULL = the null stream).  workspace: at least lcsm_base_workspace_bytes
 * bytes, 256-byte aligned, owned by the caller; NULL makes the library
 * allocate it.  Errors: LCSM_EINVAL, LCSM_ENOMEM, LCSM_EDEVICE. */
int lcsm_base_init(lcsm_base** out, int kind, const float* filters, int M, int B, int D, int L,
                   void* stream, void* workspace, size_t workspace_bytes);

/* One position for all layers: y_t device [M][B][D] in, z_t device
 * [M][B][D] out (z_t = fmaf(h_0, y_t, sum of the earlier contributions)).
 * Errors: LCSM_EDONE once t = L, LCSM_ESTATE after a fault, LCSM_EINVAL for
 * null pointers, LCSM_EDEVICE. */
int lcsm_base_step(lcsm_base* ctx, const float* y_t, float* z_t);

/* Position 0 with the state zero (a fill kernel, no memset).  Errors:
 * LCSM_EINVAL, LCSM_EDEVICE. */
int lcsm_base_reset(lcsm_base* ctx);

/* Current position (host only). */
int lcsm_base_position(const lcsm_base* ctx, int* t);

/* Release the context (waits for its stream); NULL is ignored. */
void lcsm_base_destroy(lcsm_base* ctx);

/* Text of the last error recorded on this context ("" if none). */
const char* lcsm_base_last_error(const lcsm_base* ctx);

#ifdef __cplusplus
}
#endif

#endif /* LCSM_BASE_H */
