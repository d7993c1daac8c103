/*
 * lcsm_synth.h -- C ABI of the synthetic end-to-end model on top of the
 * relaxed online long convolution (include lcsm.h for the error codes and
 * lcsm_options).
 *
 * The model is the synthetic setup of the experiments (Sec. 5 of Oncescu et
 * al., "Flash Inference", arXiv 2410.12982), generated autoregressively as
 * in Alg. 3.  Layers m = 0..M-1 each have a long-convolution mixer (filter
 * h[m,d,k], as in lcsm_init) followed by a block, an MLP of hidden width 2D
 * with the exact GELU:
 *
 *     z^m_t     = sum_{s<=t} y^m_s[b,d] h[m,d,t-s]            (mixer m)
 *     a^{m+1}_t = W_down[m] gelu(W_up[m] z^m_t + b_up[m]) + b_down[m]
 *     y^{m+1}_t = a^{m+1}_t                                   (m+1 < M)
 *     y^0_0     = eps_0,   y^0_t = a^M_{t-1} + eps_t           (the sampler)
 *
 * with gelu(x) = x/2 (1 + erf(x / sqrt 2)).  The sampler noise eps_t is an
 * input of each step.  Per position the library runs the sampler with layer
 * 0's red cell, then per layer the two matrix-vector products (the second
 * one also doing the next layer's red cell), then the gray tiles of all
 * layers in one batch (as lcsm_step does).
 *
 * Conventions as in lcsm.h: device fp32 pointers, asynchronous on the
 * context's stream, LCSM_* return codes, arguments validated before any
 * device work is queued, not thread safe.
 */
#ifndef LCSM_SYNTH_H
#define LCSM_SYNTH_H

#include <stddef.h>

#include "lcsm.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lcsm_synth lcsm_synth;

/* Create a model context.
 *   filters  device [M][D][L] fp32 (as lcsm_init);
 *   w_up     device [M][2D][D] fp32, the first layer of each block in the
 *            [out][in] layout (row n holds the weights of hidden unit n);
 *   b_up     device [M][2D];
 *   w_down   device [M][D][2D] ([out][in]);  b_down  device [M][D].
 * All five are copied during the call's stream work; the caller may free
 * them once the stream has passed lcsm_synth_init.  D must be a multiple of
 * 4 (16-byte weight rows).  opt is passed to the mixer (lcsm_options,
 * NULL for the defaults).  The library allocates its device memory (the
 * mixer's workspace, a copy of the weights, M*(4D*D + 3D) floats, and
 * (4 B D) floats of buffers).  Errors: LCSM_EINVAL (null pointers, D not a
 * multiple of 4, or what lcsm_init rejects), LCSM_ENOMEM, LCSM_EDEVICE;
 * *out is NULL on failure. */
int lcsm_synth_init(lcsm_synth** out, const float* filters, const float* w_up, const float* b_up,
                    const float* w_down, const float* b_down, int M, int B, int D, int L,
                    void* stream, const lcsm_options* opt);

/* One position t of the model:
 *   eps_t  device [B][D]: the sampler noise of position t;
 *   act_t  device [M][B][D]: receives the block outputs a^{m+1}_t of every
 *          layer (act_t[M-1] = a^M_t, the model's output at t).
 * Advances t.  eps_t and act_t may not overlap.  Errors: LCSM_EDONE once
 * t = L, LCSM_ESTATE after a fault, LCSM_EINVAL for null pointers,
 * LCSM_EDEVICE. */
int lcsm_synth_step(lcsm_synth* s, const float* eps_t, float* act_t);

/* Back to position 0 (all activations zero); keeps filters and weights and
 * clears a fault.  Errors: LCSM_EDEVICE. */
int lcsm_synth_reset(lcsm_synth* s);

/* Current position t (the next step emits position t).  Host only. */
int lcsm_synth_position(const lcsm_synth* s, int* t);

/* Release the context (waits for its stream).  NULL is ignored. */
void lcsm_synth_destroy(lcsm_synth* s);

/* Text of the last error recorded on this context ("" if none). */
const char* lcsm_synth_last_error(const lcsm_synth* s);

#ifdef __cplusplus
}
#endif

#endif /* LCSM_SYNTH_H */
