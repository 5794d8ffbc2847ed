// evo_proj_api.cpp -- the C ABI declared in include/evo_proj.h: validation
// (before any HIP call) and dispatch.
#include "evo_proj.h"

#include <hip/hip_runtime.h>
#include <math.h>

#include "evo_kernels.h"

namespace {

bool aligned(const void *p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

}  // namespace

extern "C" {

namespace {

int check_proj(const evo_proj_dims *d) {
    if (!d || d->reserved != 0) return EVO_ERR_INVALID_ARG;
    if (d->dtype != EVO_DTYPE_BF16) return EVO_ERR_UNSUPPORTED;
    if (d->n_rows < 0 || d->c_in < 1 || d->n_proj < 1 || d->proj_dim < 1 || !(d->eps >= 0.0f) ||
        !isfinite(d->eps))
        return EVO_ERR_INVALID_ARG;
    if (!evo::proj_supported(d->c_in, d->proj_dim, d->n_proj)) return EVO_ERR_UNSUPPORTED;
    if (d->n_rows > (int64_t(1) << 36)) return EVO_ERR_UNSUPPORTED;
    return EVO_OK;
}

}  // namespace

int evo_ln_proj_fwd(const evo_proj_dims *d, const void *x, const float *ln_weight, const float *ln_bias,
                    const void *weight, const float *bias, void *const *outs, float *mean, float *rstd,
                    void *stream) {
    return evo_ln_proj_fwd_ex(d, x, ln_weight, ln_bias, weight, bias, outs, mean, rstd, nullptr, stream);
}

int evo_ln_proj_fwd_ex(const evo_proj_dims *d, const void *x, const float *ln_weight, const float *ln_bias,
                       const void *weight, const float *bias, void *const *outs, float *mean, float *rstd,
                       void *y_norm, void *stream) {
    const int st = check_proj(d);
    if (st) return st;
    if (d->n_rows == 0) return EVO_OK;
    if (!x || !ln_weight || !ln_bias || !weight || !outs) return EVO_ERR_INVALID_ARG;
    if ((mean == nullptr) != (rstd == nullptr) || (mean && (void *)mean == (void *)rstd)) return EVO_ERR_INVALID_ARG;
    if (y_norm && (y_norm == x || !aligned(y_norm, 16))) return y_norm == x ? EVO_ERR_INVALID_ARG : EVO_ERR_ALIGNMENT;
    for (int p = 0; p < d->n_proj; ++p) {
        if (!outs[p] || outs[p] == x || outs[p] == weight || outs[p] == y_norm) return EVO_ERR_INVALID_ARG;
        for (int q = 0; q < p; ++q)
            if (outs[q] == outs[p]) return EVO_ERR_INVALID_ARG;
        if (!aligned(outs[p], 16)) return EVO_ERR_ALIGNMENT;
    }
    if (!aligned(x, 16) || !aligned(weight, 16) || !aligned(ln_weight, 16) || !aligned(ln_bias, 16) ||
        (bias && !aligned(bias, 16)) || (mean && (!aligned(mean, 4) || !aligned(rstd, 4))))
        return EVO_ERR_ALIGNMENT;
    evo::PjArgs a{};
    a.x = x;
    a.lnw = ln_weight;
    a.lnb = ln_bias;
    a.W = weight;
    a.bias = bias;
    void *o[4] = {outs[0], d->n_proj > 1 ? outs[1] : nullptr, d->n_proj > 2 ? outs[2] : nullptr,
                  d->n_proj > 3 ? outs[3] : nullptr};
    a.out0 = o[0];
    a.out1 = o[1];
    a.out2 = o[2];
    a.out3 = o[3];
    a.mean = mean;
    a.rstd = rstd;
    a.y = y_norm;
    a.R = d->n_rows;
    a.C = d->c_in;
    a.HD = d->proj_dim;
    a.P = d->n_proj;
    a.eps = d->eps;
    return evo::launch_ln_proj(a, (hipStream_t)stream) == hipSuccess ? EVO_OK : EVO_ERR_HIP;
}

size_t evo_ln_proj_bwd_workspace_size(const evo_proj_dims *d) {
    if (check_proj(d)) return 0;
    return evo::plan_proj_bwd(d->n_rows, d->c_in, d->proj_dim, d->n_proj).total;
}

int evo_ln_proj_bwd(const evo_proj_dims *d, const void *x, const float *ln_weight, const float *mean,
                    const float *rstd, const void *y_norm, const void *weight, const void *const *douts, void *dx,
                    float *dweight, float *dbias, float *dln_weight, float *dln_bias, void *workspace,
                    size_t workspace_bytes, void *stream) {
    int st = check_proj(d);
    if (st) return st;
    if (d->n_rows == 0) return EVO_OK;
    if (!x || !ln_weight || !mean || !rstd || !y_norm || !weight || !douts || !dx || !dweight || !dln_weight ||
        !dln_bias)
        return EVO_ERR_INVALID_ARG;
    for (int p = 0; p < d->n_proj; ++p) {
        if (!douts[p]) return EVO_ERR_INVALID_ARG;
        if (!aligned(douts[p], 16)) return EVO_ERR_ALIGNMENT;
    }
    if (dx == x || dx == y_norm || (void *)dln_weight == (void *)dln_bias) return EVO_ERR_INVALID_ARG;
    const void *al16[] = {x, y_norm, weight, dx, dweight, dln_weight, dln_bias, ln_weight};
    for (const void *q : al16)
        if (!aligned(q, 16)) return EVO_ERR_ALIGNMENT;
    if ((dbias && !aligned(dbias, 16)) || !aligned(mean, 4) || !aligned(rstd, 4)) return EVO_ERR_ALIGNMENT;
    const evo::PjBwdPlan plan = evo::plan_proj_bwd(d->n_rows, d->c_in, d->proj_dim, d->n_proj);
    if (!workspace || workspace_bytes < plan.total || !aligned(workspace, 256)) return EVO_ERR_WORKSPACE;
    evo::PjBwdArgs a{};
    a.x = x;
    a.lnw = ln_weight;
    a.mean = mean;
    a.rstd = rstd;
    a.y = y_norm;
    a.W = weight;
    a.dout0 = douts[0];
    a.dout1 = d->n_proj > 1 ? douts[1] : nullptr;
    a.dout2 = d->n_proj > 2 ? douts[2] : nullptr;
    a.dout3 = d->n_proj > 3 ? douts[3] : nullptr;
    a.dx = dx;
    a.dW = dweight;
    a.dbias = dbias;
    a.dlnw = dln_weight;
    a.dlnb = dln_bias;
    a.R = d->n_rows;
    a.C = d->c_in;
    a.HD = d->proj_dim;
    a.P = d->n_proj;
    return evo::launch_ln_proj_bwd(a, workspace, plan, (hipStream_t)stream) == hipSuccess ? EVO_OK : EVO_ERR_HIP;
}

int evo_linear_fwd(const evo_proj_dims *d, const void *x, const void *weight, const float *bias, void *const *outs,
                   void *stream) {
    const int st = check_proj(d);
    if (st) return st;
    if (d->n_rows == 0) return EVO_OK;
    if (!x || !weight || !outs) return EVO_ERR_INVALID_ARG;
    for (int p = 0; p < d->n_proj; ++p) {
        if (!outs[p] || outs[p] == x || outs[p] == weight) return EVO_ERR_INVALID_ARG;
        for (int q = 0; q < p; ++q)
            if (outs[q] == outs[p]) return EVO_ERR_INVALID_ARG;
        if (!aligned(outs[p], 16)) return EVO_ERR_ALIGNMENT;
    }
    if (!aligned(x, 16) || !aligned(weight, 16) || (bias && !aligned(bias, 16))) return EVO_ERR_ALIGNMENT;
    evo::PjArgs a{};
    a.x = x;
    a.W = weight;
    a.bias = bias;
    a.out0 = outs[0];
    a.out1 = d->n_proj > 1 ? outs[1] : nullptr;
    a.out2 = d->n_proj > 2 ? outs[2] : nullptr;
    a.out3 = d->n_proj > 3 ? outs[3] : nullptr;
    a.R = d->n_rows;
    a.C = d->c_in;
    a.HD = d->proj_dim;
    a.P = d->n_proj;
    a.eps = d->eps;
    return evo::launch_ln_proj(a, (hipStream_t)stream) == hipSuccess ? EVO_OK : EVO_ERR_HIP;
}

size_t evo_linear_bwd_workspace_size(const evo_proj_dims *d) {
    if (check_proj(d)) return 0;
    return evo::plan_proj_bwd(d->n_rows, d->c_in, d->proj_dim, d->n_proj, false).total;
}

int evo_linear_bwd(const evo_proj_dims *d, const void *x, const void *weight, const void *const *douts, void *dx,
                   float *dweight, float *dbias, void *workspace, size_t workspace_bytes, void *stream) {
    const int st = check_proj(d);
    if (st) return st;
    if (d->n_rows == 0) return EVO_OK;
    if (!x || !weight || !douts || !dx || !dweight) return EVO_ERR_INVALID_ARG;
    for (int p = 0; p < d->n_proj; ++p) {
        if (!douts[p]) return EVO_ERR_INVALID_ARG;
        if (!aligned(douts[p], 16)) return EVO_ERR_ALIGNMENT;
    }
    if (dx == x || (void *)dweight == (void *)dbias) return EVO_ERR_INVALID_ARG;
    const void *al16[] = {x, weight, dx, dweight};
    for (const void *q : al16)
        if (!aligned(q, 16)) return EVO_ERR_ALIGNMENT;
    if (dbias && !aligned(dbias, 16)) return EVO_ERR_ALIGNMENT;
    const evo::PjBwdPlan plan = evo::plan_proj_bwd(d->n_rows, d->c_in, d->proj_dim, d->n_proj, false);
    if (!workspace || workspace_bytes < plan.total || !aligned(workspace, 256)) return EVO_ERR_WORKSPACE;
    evo::PjBwdArgs a{};
    a.x = x;
    a.y = x;
    a.W = weight;
    a.dout0 = douts[0];
    a.dout1 = d->n_proj > 1 ? douts[1] : nullptr;
    a.dout2 = d->n_proj > 2 ? douts[2] : nullptr;
    a.dout3 = d->n_proj > 3 ? douts[3] : nullptr;
    a.dx = dx;
    a.dW = dweight;
    a.dbias = dbias;
    a.R = d->n_rows;
    a.C = d->c_in;
    a.HD = d->proj_dim;
    a.P = d->n_proj;
    return evo::launch_ln_proj_bwd(a, workspace, plan, (hipStream_t)stream) == hipSuccess ? EVO_OK : EVO_ERR_HIP;
}

// dims shared by the pair-bias forward and backward; `bwd` also requires the
// backward's compiled head counts and its fp32 gradient plane below 2^31 bytes
static int check_pb(const evo_pair_bias_dims *d, bool bwd) {
    if (!d || d->reserved != 0) return EVO_ERR_INVALID_ARG;
    if (d->dtype != EVO_DTYPE_BF16) return EVO_ERR_UNSUPPORTED;
    if (d->n_batch < 0 || d->len_i < 0 || d->len_j < 0 || d->c_in < 1 || d->n_heads < 1 ||
        (d->transpose != 0 && d->transpose != 1) || !(d->eps >= 0.0f) || !isfinite(d->eps))
        return EVO_ERR_INVALID_ARG;
    if (!(bwd ? evo::pair_bias_bwd_supported(d->c_in, d->n_heads) : evo::pair_bias_supported(d->c_in, d->n_heads)))
        return EVO_ERR_UNSUPPORTED;
    if (d->len_i % 8 != 0 || d->len_j % 8 != 0) return EVO_ERR_UNSUPPORTED;
    if ((int64_t)d->n_heads * d->len_i * d->len_j * (bwd ? 4 : 2) >= 0x7fffffffLL ||
        d->len_j * d->c_in * 2 >= 0x7fffffffLL || d->n_batch > 65535)
        return EVO_ERR_UNSUPPORTED;
    return EVO_OK;
}

int evo_ln_pair_bias_fwd(const evo_pair_bias_dims *d, const void *z, const float *ln_weight, const float *ln_bias,
                         const void *weight, void *out, float *mean, float *rstd, void *stream) {
    const int st = check_pb(d, false);
    if (st) return st;
    if (d->n_batch == 0 || d->len_i == 0 || d->len_j == 0) return EVO_OK;
    if (!z || !ln_weight || !ln_bias || !weight || !out || out == z) return EVO_ERR_INVALID_ARG;
    if ((mean == nullptr) != (rstd == nullptr) || (mean && (void *)mean == (void *)rstd)) return EVO_ERR_INVALID_ARG;
    if (!aligned(z, 16) || !aligned(weight, 16) || !aligned(out, 16) || !aligned(ln_weight, 16) ||
        !aligned(ln_bias, 16) || (mean && (!aligned(mean, 4) || !aligned(rstd, 4))))
        return EVO_ERR_ALIGNMENT;
    evo::PbArgs a{};
    a.z = z;
    a.lnw = ln_weight;
    a.lnb = ln_bias;
    a.W = weight;
    a.out = out;
    a.mean = mean;
    a.rstd = rstd;
    a.B = d->n_batch;
    a.Li = (int)d->len_i;
    a.Lj = (int)d->len_j;
    a.C = d->c_in;
    a.H = d->n_heads;
    a.transpose = d->transpose;
    a.eps = d->eps;
    return evo::launch_pair_bias(a, (hipStream_t)stream) == hipSuccess ? EVO_OK : EVO_ERR_HIP;
}

size_t evo_ln_pair_bias_bwd_workspace_size(const evo_pair_bias_dims *d) {
    if (check_pb(d, true) || d->n_batch == 0 || d->len_i == 0 || d->len_j == 0) return 0;
    return evo::pair_bias_bwd_workspace(d->n_batch, (int)d->len_i, (int)d->len_j, d->c_in, d->n_heads);
}

int evo_ln_pair_bias_bwd(const evo_pair_bias_dims *d, const void *z, const float *ln_weight, const float *ln_bias,
                         const void *weight, const float *dbias, void *dz, float *dweight, float *dln_weight,
                         float *dln_bias, void *workspace, size_t workspace_bytes, void *stream) {
    const int st = check_pb(d, true);
    if (st) return st;
    if (d->n_batch == 0 || d->len_i == 0 || d->len_j == 0) return EVO_OK;
    if (!z || !ln_weight || !ln_bias || !weight || !dbias || !dz || !dweight || !dln_weight || !dln_bias)
        return EVO_ERR_INVALID_ARG;
    if (dz == z || (const void *)dz == (const void *)dbias || dweight == dln_weight || dweight == dln_bias ||
        dln_weight == dln_bias)
        return EVO_ERR_INVALID_ARG;
    const void *al16[] = {z, ln_weight, ln_bias, weight, dbias, dz, dweight, dln_weight, dln_bias};
    for (const void *p : al16)
        if (!aligned(p, 16)) return EVO_ERR_ALIGNMENT;
    const size_t need = evo::pair_bias_bwd_workspace(d->n_batch, (int)d->len_i, (int)d->len_j, d->c_in, d->n_heads);
    if (!workspace || workspace_bytes < need) return EVO_ERR_WORKSPACE;
    if (!aligned(workspace, 16)) return EVO_ERR_ALIGNMENT;
    evo::PbBwdArgs a{};
    a.z = z;
    a.lnw = ln_weight;
    a.lnb = ln_bias;
    a.W = weight;
    a.dbias = dbias;
    a.dz = dz;
    a.dW = dweight;
    a.dlnw = dln_weight;
    a.dlnb = dln_bias;
    a.B = d->n_batch;
    a.Li = (int)d->len_i;
    a.Lj = (int)d->len_j;
    a.C = d->c_in;
    a.H = d->n_heads;
    a.transpose = d->transpose;
    a.eps = d->eps;
    return evo::launch_pair_bias_bwd(a, workspace, (hipStream_t)stream) == hipSuccess ? EVO_OK : EVO_ERR_HIP;
}

}  // extern "C"
