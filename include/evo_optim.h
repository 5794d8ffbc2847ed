/*
 * evo_optim.h -- C ABI of the fused optimizer step on MI355X (gfx950):
 * gradient-norm clipping, Adam and the stochastic weight average (SWA) over
 * a packed list of parameter tensors.
 *
 * ScaleFold (arXiv 2404.11068), Section 3.3, "Adam and SWA Optimization":
 * Adam, the SWA update that follows it and the adjacent elementwise work run
 * as one kernel over all parameters, each thread block on a contiguous
 * sub-region, with the pointers of every parameter and optimizer-state
 * tensor packed into one buffer so that a single launch covers them all;
 * "Gradient Clipping Optimization": the gradient norm is computed over the
 * packed gradients instead of one launch per tensor.  Per element (fp32):
 *
 *   g  = grad * scale  (+ weight_decay * p if weight_decay != 0)
 *   m  = beta1 m + (1 - beta1) g
 *   v  = beta2 v + (1 - beta2) g^2
 *   p  = p - lr * (m / (1 - beta1^step)) / (sqrt(v / (1 - beta2^step)) + eps)
 *   w  = swa_decay * w + (1 - swa_decay) * p        (skipped when swa == NULL)
 *
 * and the clipping scale over all gradient elements:
 *
 *   norm = sqrt(sum g^2),  scale = min(1, max_norm / (norm + 1e-6))
 *
 * Tables: the caller packs one evo_mt_tensor per parameter and the list of
 * evo_mt_chunk work items (EVO_MT_CHUNK elements each; evo_mt_build_chunks
 * fills it on the host) into DEVICE memory and passes both; they depend on
 * the tensor sizes only, so they are built once and reused every step.
 * Entries whose tensor index is out of range or whose chunk lies past the
 * tensor's end are skipped by the kernels.  All tensor pointers are device
 * pointers (fp32); 16-byte aligned pointers take the vector path, others a
 * slower per-element path.  Nothing is allocated or synchronised; the calls
 * only enqueue kernels on `stream`.  Status codes are those of evo_attn.h.
 */
#ifndef EVO_OPTIM_H
#define EVO_OPTIM_H

#include "evo_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

#define EVO_MT_CHUNK 4096

typedef struct evo_mt_tensor {
    float *param;        /* updated in place */
    const float *grad;   /* read only */
    float *exp_avg;      /* m, updated in place */
    float *exp_avg_sq;   /* v, updated in place */
    float *swa;          /* averaged parameters, updated in place; NULL = no SWA */
    int64_t numel;       /* elements, >= 0 */
} evo_mt_tensor;

typedef struct evo_mt_chunk {
    int32_t tensor;      /* index into the tensor table */
    int32_t index;       /* elements [index * EVO_MT_CHUNK, min(numel, (index + 1) * EVO_MT_CHUNK)) */
} evo_mt_chunk;

/* Hyperparameters in double: the library derives 1 - beta, the bias
 * corrections 1 - beta^step and 1 - swa_decay in double and rounds each
 * once to fp32 (rounding beta2 = 0.999 to fp32 first would move 1 - beta2
 * and 1 - beta2^step by about 1e-5 relative). */
typedef struct evo_adam_swa_hparams {
    double lr, beta1, beta2, eps, weight_decay, swa_decay;
    int64_t step;        /* >= 1: the bias corrections use beta^step */
} evo_adam_swa_hparams;

/* Host helper: number of chunks for these tensor sizes (-1 if a size is
 * negative or the count exceeds 2^31 - 1). */
int64_t evo_mt_chunk_count(const int64_t *numels, int32_t n_tensors);

/* Host helper: writes the chunk list (host memory, `capacity` entries) in
 * tensor order; returns the number written or -1 (bad sizes or capacity). */
int64_t evo_mt_build_chunks(const int64_t *numels, int32_t n_tensors, evo_mt_chunk *out, int64_t capacity);

/* Gradient norm and clipping scale over every gradient of the table.
 * workspace: device fp32 array of at least n_chunks entries (per-chunk sums,
 * contents on entry irrelevant); norm_out, scale_out: device fp32 scalars
 * (either may be NULL).  Sums are taken in a fixed order (repeatable). */
int evo_grad_clip_scale(const evo_mt_tensor *tensors, int32_t n_tensors, const evo_mt_chunk *chunks,
                        int32_t n_chunks, float max_norm, float *workspace, float *norm_out,
                        float *scale_out, void *stream);

/* One fused Adam + SWA step.  grad_scale: device fp32 scalar multiplying
 * every gradient (e.g. scale_out of evo_grad_clip_scale) or NULL for 1. */
int evo_adam_swa_step(const evo_adam_swa_hparams *hp, const evo_mt_tensor *tensors, int32_t n_tensors,
                      const evo_mt_chunk *chunks, int32_t n_chunks, const float *grad_scale, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* EVO_OPTIM_H */
