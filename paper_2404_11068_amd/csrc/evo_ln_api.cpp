// evo_ln_api.cpp -- the C ABI declared in include/evo_layernorm.h: argument
// validation (before any HIP call) and kernel dispatch.
#include "evo_layernorm.h"

#include <hip/hip_runtime.h>
#include <math.h>

#include "evo_kernels.h"

namespace {

bool aligned(const void *p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

int check_ln(const evo_ln_dims *d, evo::LnProblem *p) {
    if (!d || d->reserved != 0) return EVO_ERR_INVALID_ARG;
    if (d->dtype != EVO_DTYPE_F32 && d->dtype != EVO_DTYPE_BF16) return EVO_ERR_UNSUPPORTED;
    if (d->n_rows < 0 || d->n_cols < 1 || !(d->eps >= 0.0f) || !isfinite(d->eps)) return EVO_ERR_INVALID_ARG;
    if (!evo::ln_supported_cols(d->n_cols)) return EVO_ERR_UNSUPPORTED;
    const int es = d->dtype == EVO_DTYPE_BF16 ? 2 : 4;
    if (d->n_rows > (int64_t(1) << 40) / ((int64_t)d->n_cols * es)) return EVO_ERR_UNSUPPORTED;
    p->dtype = d->dtype;
    p->C = d->n_cols;
    p->R = d->n_rows;
    p->eps = d->eps;
    return EVO_OK;
}

}  // namespace

extern "C" {

int evo_layernorm_fwd(const evo_ln_dims *dims, const void *x, const float *weight, const float *bias, void *y,
                      float *mean, float *rstd, void *stream) {
    evo::LnProblem p;
    int st = check_ln(dims, &p);
    if (st) return st;
    if (p.R == 0) return EVO_OK;
    if (!x || !weight || !bias || !y) return EVO_ERR_INVALID_ARG;
    if (y == x || (mean && (void *)mean == (void *)rstd)) return EVO_ERR_INVALID_ARG;
    if (!aligned(x, 16) || !aligned(y, 16) || !aligned(weight, 16) || !aligned(bias, 16) ||
        (mean && !aligned(mean, 4)) || (rstd && !aligned(rstd, 4)))
        return EVO_ERR_ALIGNMENT;
    evo::LnPtrs ptr{x, weight, bias, y, mean, rstd};
    return evo::launch_ln_fwd(p, ptr, (hipStream_t)stream) == hipSuccess ? EVO_OK : EVO_ERR_HIP;
}

size_t evo_layernorm_bwd_workspace_size(const evo_ln_dims *dims) {
    evo::LnProblem p;
    if (check_ln(dims, &p)) return 0;
    return evo::ln_bwd_workspace(p);
}

namespace {

int ln_bwd_impl(const evo_ln_dims *dims, const void *x, const float *weight, const float *mean, const float *rstd,
                const void *dy, void *dx, float *dweight, float *dbias, void *workspace, size_t workspace_bytes,
                void *stream, evo::Tracer *tr) {
    evo::LnProblem p;
    int st = check_ln(dims, &p);
    if (st) return st;
    if (!dweight || !dbias || dweight == dbias) return EVO_ERR_INVALID_ARG;
    if (!aligned(dweight, 16) || !aligned(dbias, 16)) return EVO_ERR_ALIGNMENT;
    if (p.R > 0) {
        if (!x || !weight || !mean || !rstd || !dy || !dx) return EVO_ERR_INVALID_ARG;
        if (dx == x || dx == dy) return EVO_ERR_INVALID_ARG;
        if (!aligned(x, 16) || !aligned(dy, 16) || !aligned(dx, 16) || !aligned(weight, 16) ||
            !aligned(mean, 4) || !aligned(rstd, 4))
            return EVO_ERR_ALIGNMENT;
        if (!workspace || workspace_bytes < evo::ln_bwd_workspace(p) || !aligned(workspace, 256))
            return EVO_ERR_WORKSPACE;
    }
    if (tr) {
        if (tr->n < 3) return EVO_ERR_INVALID_ARG;
        for (int i = 0; i < tr->n; ++i)
            if (!tr->ev[i]) return EVO_ERR_INVALID_ARG;
    }
    evo::LnBwdPtrs ptr{x, weight, mean, rstd, dy, dx, dweight, dbias};
    return evo::launch_ln_bwd(p, ptr, workspace, (hipStream_t)stream, tr) == hipSuccess ? EVO_OK : EVO_ERR_HIP;
}

}  // namespace

int evo_layernorm_bwd(const evo_ln_dims *dims, const void *x, const float *weight, const float *mean,
                      const float *rstd, const void *dy, void *dx, float *dweight, float *dbias, void *workspace,
                      size_t workspace_bytes, void *stream) {
    return ln_bwd_impl(dims, x, weight, mean, rstd, dy, dx, dweight, dbias, workspace, workspace_bytes, stream,
                       nullptr);
}

int evo_layernorm_bwd_traced(const evo_ln_dims *dims, const void *x, const float *weight, const float *mean,
                             const float *rstd, const void *dy, void *dx, float *dweight, float *dbias,
                             void *workspace, size_t workspace_bytes, void *const *events, int n_events,
                             void *stream) {
    if (!events || n_events < 1) return EVO_ERR_INVALID_ARG;
    evo::Tracer tr;
    tr.ev = (hipEvent_t const *)events;
    tr.n = n_events;
    return ln_bwd_impl(dims, x, weight, mean, rstd, dy, dx, dweight, dbias, workspace, workspace_bytes, stream,
                       &tr);
}

}  // extern "C"
