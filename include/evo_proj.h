/*
 * evo_proj.h -- C ABI of the fused LayerNorm + batched projections (gfx950).
 *
 * The step in front of every Evoformer attention: normalise the input
 * representation and project it to queries, keys, values and gate logits.
 * ScaleFold (arXiv 2404.11068), Section 3.3, GEMM Batching: the query, key,
 * value and gate projections read the same input and none needs another's
 * result, so they run as one batched product, fused here with the LayerNorm
 * in front of them.  Computed here:
 *
 *   y        = LayerNorm(x) over the last axis (as in evo_layernorm.h), bf16
 *   out_p    = y @ weight[p*HD : (p+1)*HD, :]^T + bias[p*HD : (p+1)*HD]
 *              for p = 0 .. n_proj-1
 *
 * Each out_p is written straight into the attention's token layout: a
 * contiguous [R, HD] bf16 tensor is the [N, L, H, d] tensor with R = N*L and
 * HD = H*d, ready for evo_attn_fwd.
 *
 * Conventions (dtype and status codes from evo_attn.h):
 * - Device pointers owned by the caller; nothing is allocated or
 *   synchronised; the call enqueues one kernel on `stream` and returns.
 * - x: contiguous [R, C] bf16, 16-byte aligned.  ln_weight, ln_bias: fp32
 *   [C].  weight: contiguous [n_proj*HD, C] bf16 (torch Linear layout,
 *   projections stacked), 16-byte aligned.  bias: fp32 [n_proj*HD] or NULL.
 *   outs: HOST array of n_proj device pointers, each a contiguous [R, HD]
 *   bf16 tensor, 16-byte aligned, not aliasing each other or any input.
 *   mean, rstd: fp32 [R] LayerNorm statistics (both or neither; NULL = not
 *   stored).
 * - The LayerNorm output is rounded to bf16 before the products (the MFMA
 *   input precision); products accumulate in fp32; outputs are rounded to
 *   nearest even.
 * - Validation happens before any HIP call; errors enqueue nothing.
 */
#ifndef EVO_PROJ_H
#define EVO_PROJ_H

#include "evo_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Compiled set: dtype EVO_DTYPE_BF16; c_in in {64, 128, 256}; proj_dim a
 * multiple of 32 in [32, 1024]; n_proj in [1, 4]. */
typedef struct evo_proj_dims {
    int32_t dtype;     /* EVO_DTYPE_BF16 */
    int32_t c_in;      /* C */
    int32_t n_proj;    /* P */
    int32_t proj_dim;  /* HD = H * d per projection */
    int64_t n_rows;    /* R >= 0 tokens (N * L) */
    float eps;         /* LayerNorm epsilon, >= 0 and finite */
    int32_t reserved;  /* must be 0 */
} evo_proj_dims;

/* R == 0 validates and returns EVO_OK without touching any pointer. */
int evo_ln_proj_fwd(const evo_proj_dims *dims, const void *x, const float *ln_weight,
                    const float *ln_bias, const void *weight, const float *bias,
                    void *const *outs, float *mean, float *rstd, void *stream);

/* Training variant: as evo_ln_proj_fwd, and when y_norm is not NULL also
 * writes the normalised input LayerNorm(x) as rounded to bf16 for the
 * products (contiguous [R, C] bf16, 16-byte aligned), which the backward
 * reads. */
int evo_ln_proj_fwd_ex(const evo_proj_dims *dims, const void *x, const float *ln_weight,
                       const float *ln_bias, const void *weight, const float *bias,
                       void *const *outs, float *mean, float *rstd, void *y_norm, void *stream);

/*
 * Backward of the fused LayerNorm + projections.  With y = y_norm (the
 * forward's normalised input) and upstream gradients douts[p] ([R, HD] bf16,
 * a HOST array of n_proj device pointers):
 *
 *   dY       = sum_p douts[p] @ weight[p*HD:(p+1)*HD, :]   rounded to bf16
 *   dx, dln_weight, dln_bias = LayerNorm backward of dY (as evo_layernorm_bwd,
 *              from x, ln_weight and the forward's mean, rstd)
 *   dweight[p*HD + f, c] = sum_t douts[p][t, f] * y[t, c]   (fp32)
 *   dbias[p*HD + f]      = sum_t douts[p][t, f]             (fp32; NULL: not computed)
 *
 * dx: [R, C] bf16 output; dweight: [n_proj*HD, C] fp32; dbias: [n_proj*HD]
 * fp32 or NULL; dln_weight, dln_bias: [C] fp32 (all 16-byte aligned).
 * workspace: at least evo_ln_proj_bwd_workspace_size(dims) bytes, 256-byte
 * aligned, contents irrelevant.  Every sum runs in a fixed order (repeatable
 * results).  R == 0 validates and returns EVO_OK without touching anything.
 */
size_t evo_ln_proj_bwd_workspace_size(const evo_proj_dims *dims);
int evo_ln_proj_bwd(const evo_proj_dims *dims, const void *x, const float *ln_weight, const float *mean,
                    const float *rstd, const void *y_norm, const void *weight, const void *const *douts,
                    void *dx, float *dweight, float *dbias, float *dln_weight, float *dln_bias,
                    void *workspace, size_t workspace_bytes, void *stream);

/*
 * Linear layers without the LayerNorm: the same batched products on x itself,
 * outs[p] = x @ weight[p*HD:(p+1)*HD, :]^T + bias[p*HD:(p+1)*HD] — the output
 * projection that follows the gated attention in every Evoformer attention
 * module (ScaleFold Section 3.3 fuses the module's other linear layers with
 * its LayerNorm and MHA; this one reads the attention's gated output, [N, L,
 * H, d] = [R, C] with C = H * d).  dims, layouts and compiled set as above;
 * eps is unused (still validated).
 *
 * Backward: dx = sum_p douts[p] @ weight_p (rounded to bf16, written to dx),
 * dweight[p*HD + f, c] = sum_t douts[p][t, f] * x[t, c], dbias as above.
 * workspace: evo_linear_bwd_workspace_size(dims) bytes, 256-byte aligned.
 * Errors as for the LayerNorm variants; R == 0 returns EVO_OK untouched.
 */
int evo_linear_fwd(const evo_proj_dims *dims, const void *x, const void *weight, const float *bias,
                   void *const *outs, void *stream);
size_t evo_linear_bwd_workspace_size(const evo_proj_dims *dims);
int evo_linear_bwd(const evo_proj_dims *dims, const void *x, const void *weight, const void *const *douts,
                   void *dx, float *dweight, float *dbias, void *workspace, size_t workspace_bytes,
                   void *stream);

/*
 * Pair bias: the logit bias every pair-biased Evoformer attention adds before
 * its softmax (ScaleFold Section 3.3, "Multi Head Attention"), a LayerNorm of
 * each pair entry followed by a bias-free linear map to one value per head,
 * written straight into the [B, H, L, L] layout evo_attn_fwd reads:
 *
 *   y          = LayerNorm(z[b, i, j, :])   (fp32 statistics, rounded to bf16)
 *   v[h]       = sum_c y[c] * weight[h, c]  (fp32 accumulation)
 *   transpose == 0:  out[b, h, i, j] = v[h]        out is [B, H, Li, Lj]
 *   transpose == 1:  out[b, h, j, i] = v[h]        out is [B, H, Lj, Li]
 *
 * (the transposed layout is the bias of triangle attention around the ending
 * node, which attends over the transposed pair representation).
 *
 * z: contiguous [B, Li, Lj, C] bf16, 16-byte aligned; ln_weight, ln_bias:
 * fp32 [C], 16-byte aligned; weight: contiguous [H, C] bf16, 16-byte aligned;
 * out: contiguous bf16 (shape above), 16-byte aligned, not aliasing z;
 * mean, rstd: fp32 [B, Li, Lj] (both or neither).
 * Compiled set: C in {64, 128, 256}; H in {1, 2, 4, 8, 16}; Li and Lj
 * multiples of 8 with H * Li * Lj * 2 bytes below 2^31.  B, Li or Lj == 0
 * validates and returns EVO_OK without touching any pointer.
 */
typedef struct evo_pair_bias_dims {
    int32_t dtype;      /* EVO_DTYPE_BF16 */
    int32_t c_in;       /* C */
    int32_t n_heads;    /* H */
    int32_t transpose;  /* 0 or 1, see above */
    int64_t n_batch;    /* B >= 0 */
    int64_t len_i;      /* Li >= 0 */
    int64_t len_j;      /* Lj >= 0 */
    float eps;          /* >= 0 and finite */
    int32_t reserved;   /* must be 0 */
} evo_pair_bias_dims;

int evo_ln_pair_bias_fwd(const evo_pair_bias_dims *dims, const void *z, const float *ln_weight,
                         const float *ln_bias, const void *weight, void *out, float *mean, float *rstd,
                         void *stream);

/* Backward of evo_ln_pair_bias_fwd (ScaleFold Section 3.3, the pair-bias term
 * of the attention, differentiated): given the attention backward's
 * dL/dbias g, in the forward's output layout (fp32 [B, H, Li, Lj], or
 * [B, H, Lj, Li] with transpose), and y = LayerNorm(z[b, i, j, :]) as above,
 *
 *   dY[b,i,j,c] = sum_h g[b,h,i,j] weight[h,c]
 *   dz          = LayerNorm backward of dY               (bf16 [B, Li, Lj, C])
 *   dweight     = sum over (b,i,j) of g[b,h,i,j] y[c]    (fp32 [H, C])
 *   dln_weight  = sum over (b,i,j) of dY * xhat,  dln_bias = sum of dY   (fp32 [C])
 *
 * The statistics are recomputed from z (the forward's are not needed).  All
 * sums run in a fixed order: repeated calls give identical bits.
 * dbias: contiguous fp32, 16-byte aligned; dz: contiguous bf16 like z,
 * 16-byte aligned, not aliasing z; dweight, dln_weight, dln_bias: fp32,
 * 16-byte aligned, distinct.  workspace: device memory of at least
 * evo_ln_pair_bias_bwd_workspace_size(dims) bytes, 16-byte aligned (nullable
 * when that size is 0), overwritten.  Compiled set: as the forward, with
 * H in {1, 2, 4, 8}.  B, Li or Lj == 0 validates and returns EVO_OK without
 * touching any pointer.  Errors: EVO_ERR_INVALID_ARG (null or aliasing
 * pointers, bad dims), EVO_ERR_UNSUPPORTED (outside the compiled set),
 * EVO_ERR_ALIGNMENT, EVO_ERR_WORKSPACE (too small), EVO_ERR_HIP (launch). */
size_t evo_ln_pair_bias_bwd_workspace_size(const evo_pair_bias_dims *dims);
int evo_ln_pair_bias_bwd(const evo_pair_bias_dims *dims, const void *z, const float *ln_weight,
                         const float *ln_bias, const void *weight, const float *dbias, void *dz,
                         float *dweight, float *dln_weight, float *dln_bias, void *workspace,
                         size_t workspace_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* EVO_PROJ_H */
