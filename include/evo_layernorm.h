/*
 * evo_layernorm.h -- C ABI of the MI355X (gfx950) LayerNorm kernels.
 *
 * Layer normalisation over the last axis, forward and backward, as it runs
 * before every Evoformer attention and transition block (MSA rows of
 * c_m = 256 channels, pair entries of c_z = 128, extra-MSA rows of c_e = 64).
 * ScaleFold (arXiv 2404.11068), Section 3.3, "LayerNormalization": the
 * paper's kernel spreads many short rows over each thread block, gets the
 * row statistics in one pass over the data, and reduces the weight and bias
 * gradients in two atomic-free steps (per-block partials, then a per-column
 * sum of the partials).  The operation itself is the usual one:
 *
 *   mean[r] = (1/C) sum_c x[r,c]
 *   rstd[r] = 1 / sqrt((1/C) sum_c (x[r,c] - mean[r])^2 + eps)
 *   y[r,c]  = (x[r,c] - mean[r]) * rstd[r] * weight[c] + bias[c]
 *
 * and its gradient, with xhat = (x - mean) * rstd and gx = dy * weight,
 *
 *   dx[r,c]   = rstd[r] * (gx[r,c] - mean_c(gx[r,:]) - xhat[r,c] * mean_c(gx[r,:] * xhat[r,:]))
 *   dweight[c] = sum_r dy[r,c] * xhat[r,c],   dbias[c] = sum_r dy[r,c]
 *
 * Conventions (shared with evo_attn.h, whose dtype and status codes these
 * entry points use):
 * - Every tensor pointer is a DEVICE pointer owned by the caller.  The
 *   library never allocates, frees or synchronises; each call only enqueues
 *   kernels on `stream` (a hipStream_t, NULL = the null stream) and returns.
 * - Process-wide state, read once: the environment variables EVO_LN_FWD_WGS
 *   and EVO_LN_BWD_WGS (positive integers) cap the forward's and the
 *   backward's workgroup counts (default: one pass per wave for the forward,
 *   512 for the backward).  Each is read on the first call that needs it,
 *   once per (dtype, channel count) kernel variant, and holds for the rest of
 *   the process; the backward's count is also its number of partial
 *   dweight/dbias rows, so set EVO_LN_BWD_WGS before the first
 *   evo_layernorm_bwd_workspace_size call.
 * - x, y, dy, dx are contiguous [R, C] in the working dtype (fp32 or bf16)
 *   and 16-byte aligned; weight, bias, dweight, dbias are contiguous fp32
 *   [C], 16-byte aligned; mean and rstd are contiguous fp32 [R], 4-byte
 *   aligned.  Statistics and all arithmetic are fp32; bf16 outputs are
 *   rounded to nearest even.
 * - Outputs are overwritten, never accumulated into, and must not alias an
 *   input.  Every sum runs in a fixed order without atomics, so repeated
 *   calls give bitwise identical results.
 * - Arguments are validated before any HIP call; an invalid call enqueues
 *   nothing and returns a nonzero evo_attn_status.
 */
#ifndef EVO_LAYERNORM_H
#define EVO_LAYERNORM_H

#include "evo_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Compiled row lengths: C in {32, 64, 128, 256, 512, 1024}. */

typedef struct evo_ln_dims {
    int32_t dtype;   /* enum evo_attn_dtype: of x, y, dy, dx */
    int32_t n_cols;  /* C, normalised axis (else EVO_ERR_UNSUPPORTED) */
    int64_t n_rows;  /* R >= 0; R * C * element size below 2^40 bytes */
    float eps;       /* >= 0 and finite, added to the variance */
    int32_t reserved; /* must be 0 */
} evo_ln_dims;

/*
 * Forward.  x: input [R,C]; weight, bias: fp32 [C] (required); y: output
 * [R,C]; mean, rstd: fp32 [R] outputs, each nullable (inference needs
 * neither; the backward needs both).  R == 0 validates and returns EVO_OK
 * without touching any pointer.
 */
int evo_layernorm_fwd(const evo_ln_dims *dims, const void *x, const float *weight, const float *bias,
                      void *y, float *mean, float *rstd, void *stream);

/*
 * Bytes of device workspace evo_layernorm_bwd needs (0 if dims is invalid):
 * one 2*C fp32 partial row per workgroup of the first step.
 */
size_t evo_layernorm_bwd_workspace_size(const evo_ln_dims *dims);

/*
 * Backward.  x, weight: as passed to the forward; mean, rstd: the forward's
 * statistics (required); dy: upstream gradient [R,C]; dx: output [R,C];
 * dweight, dbias: fp32 [C] outputs (required), summed over all R rows;
 * workspace: at least evo_layernorm_bwd_workspace_size(dims) bytes,
 * 256-byte aligned, contents on entry irrelevant (else EVO_ERR_WORKSPACE).
 * R == 0 sets dweight and dbias to zero and touches nothing else (the
 * workspace may then be NULL).
 */
int evo_layernorm_bwd(const evo_ln_dims *dims, const void *x, const float *weight, const float *mean,
                      const float *rstd, const void *dy, void *dx, float *dweight, float *dbias,
                      void *workspace, size_t workspace_bytes, void *stream);

/*
 * Profiling variant of evo_layernorm_bwd (identical arguments and results).
 * The library records the caller's hipEvent_t handles on `stream`: events[0]
 * before its first kernel and events[i] right after its i-th kernel (in this
 * version: 1 = the dx / partial-sum kernel, 2 = the per-column reduction; with
 * R == 0 only the reduction runs and events[1] is recorded before it).
 * n_events must be at least 3 and every handle non-NULL, else
 * EVO_ERR_INVALID_ARG.  Meant for benchmarks.
 */
int evo_layernorm_bwd_traced(const evo_ln_dims *dims, const void *x, const float *weight,
                             const float *mean, const float *rstd, const void *dy, void *dx,
                             float *dweight, float *dbias, void *workspace, size_t workspace_bytes,
                             void *const *events, int n_events, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* EVO_LAYERNORM_H */
