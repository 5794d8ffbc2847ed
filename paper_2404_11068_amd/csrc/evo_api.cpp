// evo_api.cpp -- the C ABI declared in include/evo_attn.h: argument
// validation (before any HIP call), workspace planning, kernel dispatch.
#include "evo_attn.h"

#include <hip/hip_runtime.h>

#include "evo_kernels.h"

namespace {

constexpr int kVersion = 10000;  // 1.0.0

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }
bool aligned4(const void *p) { return ((uintptr_t)p & 3u) == 0; }

// Common validation of dims; fills the internal problem description.
int check_dims(const evo_attn_dims *d, bool has_bias, evo::Problem *p) {
    if (!d) return EVO_ERR_INVALID_ARG;
    if (d->reserved != 0) return EVO_ERR_INVALID_ARG;
    if (d->dtype != EVO_DTYPE_F32 && d->dtype != EVO_DTYPE_BF16) return EVO_ERR_UNSUPPORTED;
    if (d->n_heads < 1 || d->head_dim < 1 || d->n_rows < 0 || d->seq_len < 0) return EVO_ERR_INVALID_ARG;
    if (d->head_dim != 8 && d->head_dim != 16 && d->head_dim != 32 && d->head_dim != 64) return EVO_ERR_UNSUPPORTED;
    if (d->seq_len > EVO_ATTN_MAX_SEQ_LEN) return EVO_ERR_UNSUPPORTED;
    if ((d->dtype == EVO_DTYPE_F32 || d->head_dim == 64) && d->seq_len > EVO_ATTN_MAX_SEQ_LEN_WIDE)
        return EVO_ERR_UNSUPPORTED;
    // fp32 at head_dim 64: the backward's LDS tiles fit up to 128 keys
    if (d->dtype == EVO_DTYPE_F32 && d->head_dim == 64 && d->seq_len > EVO_ATTN_MAX_SEQ_LEN_F32_D64)
        return EVO_ERR_UNSUPPORTED;
    const int64_t hd = (int64_t)d->n_heads * d->head_dim;
    if (d->stride_tok < hd || d->stride_row < hd) return EVO_ERR_INVALID_ARG;
    // the (row, token) grid must not overlap itself: either rows are outermost
    // (contiguous-like) or tokens are (a transposed view)
    const bool rows_outer = d->stride_row >= d->seq_len * d->stride_tok;
    const bool toks_outer = d->stride_tok >= d->n_rows * d->stride_row;
    if (!rows_outer && !toks_outer) return EVO_ERR_INVALID_ARG;
    if (has_bias) {
        if (d->rows_per_bias < 1 || d->n_rows % d->rows_per_bias != 0) return EVO_ERR_INVALID_ARG;
    }
    // grid limits of the kernels (head_dim 64 takes two workgroups per unit)
    const int64_t halves = d->head_dim > 32 ? 2 : 1;
    if ((int64_t)d->n_rows * d->n_heads * halves > 0x7fffffffLL) return EVO_ERR_UNSUPPORTED;
    if ((int64_t)d->n_rows * d->seq_len * d->n_heads * halves / 256 > 0x7fffffffLL) return EVO_ERR_UNSUPPORTED;
    const int es = d->dtype == EVO_DTYPE_BF16 ? 2 : 4;
    if ((d->stride_tok * es) % 16 != 0 || (d->stride_row * es) % 16 != 0) return EVO_ERR_ALIGNMENT;
    // the kernels address the tokens of one row with 32-bit byte offsets
    if ((int64_t)d->seq_len * d->stride_tok * es >= 0x7fffffffLL) return EVO_ERR_UNSUPPORTED;
    p->dtype = d->dtype;
    p->H = d->n_heads;
    p->D = d->head_dim;
    p->N = d->n_rows;
    p->L = d->seq_len;
    p->rpb = has_bias ? d->rows_per_bias : (d->n_rows > 0 ? d->n_rows : 1);
    p->srow = d->stride_row;
    p->stok = d->stride_tok;
    return EVO_OK;
}

}  // namespace

extern "C" {

int evo_attn_version(void) { return kVersion; }

const char *evo_attn_strerror(int status) {
    switch (status) {
        case EVO_OK: return "success";
        case EVO_ERR_INVALID_ARG: return "invalid argument (null pointer, size, rows_per_bias or strides)";
        case EVO_ERR_UNSUPPORTED: return "unsupported dtype, head_dim or seq_len";
        case EVO_ERR_ALIGNMENT: return "pointer or stride not aligned for 16-byte access";
        case EVO_ERR_WORKSPACE: return "workspace missing or too small";
        case EVO_ERR_HIP: return "HIP kernel launch failed";
        case EVO_ERR_SCRATCH_LIMIT:
            return "problem needs more backward scratch than the no-alloc entry point's fixed buffer "
                   "(EVO_ATTN_NOALLOC_SCRATCH_BYTES) holds; use evo_attn_bwd with a workspace";
        default: return "unknown status";
    }
}

int evo_attn_fwd(const evo_attn_dims *dims, const void *q, const void *k, const void *v, const void *gate,
                 const void *bias, const uint8_t *key_mask, void *out, float *lse, void *stream) {
    evo::Problem p;
    int st = check_dims(dims, bias != nullptr, &p);
    if (st) return st;
    if (p.N == 0 || p.L == 0) return EVO_OK;  // nothing is read or written
    if (!q || !k || !v || !out || !lse) return EVO_ERR_INVALID_ARG;
    if (out == q || out == k || out == v || (gate && out == gate)) return EVO_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) || (gate && !aligned16(gate)) ||
        (bias && !aligned16(bias)) || !aligned4(lse))
        return EVO_ERR_ALIGNMENT;
    evo::FwdPtrs x{q, k, v, gate, bias, key_mask, out, lse};
    hipError_t e = evo::launch_fwd(p, x, (hipStream_t)stream);
    return e == hipSuccess ? EVO_OK : EVO_ERR_HIP;
}

size_t evo_attn_bwd_workspace_size(const evo_attn_dims *dims) {
    evo::Problem p;
    // the size covers the dBias partial planes, which exist only with a bias;
    // report the larger (with-bias) plan when rows_per_bias is valid
    const bool bias_ok = dims && dims->rows_per_bias >= 1 && dims->n_rows >= 0 &&
                         dims->n_rows % (dims->rows_per_bias > 0 ? dims->rows_per_bias : 1) == 0;
    if (check_dims(dims, bias_ok, &p)) return 0;
    return evo::plan_bwd(p, bias_ok).total;
}

namespace {

// dims and pointers of a backward call (no HIP call); an empty problem
// returns EVO_OK with p->N == 0 or p->L == 0 before any pointer is looked at
int check_bwd_args(const evo_attn_dims *dims, const void *q, const void *k, const void *v, const void *gate,
                   const void *bias, const void *out, const float *lse, const void *dout, void *dq, void *dk,
                   void *dv, void *dgate, float *dbias, evo::Problem *pp) {
    evo::Problem &p = *pp;
    int st = check_dims(dims, bias != nullptr, &p);
    if (st) return st;
    if (p.N == 0 || p.L == 0) return EVO_OK;
    if (!q || !k || !v || !out || !lse || !dout || !dq || !dk || !dv) return EVO_ERR_INVALID_ARG;
    if ((gate == nullptr) != (dgate == nullptr) || (bias == nullptr) != (dbias == nullptr))
        return EVO_ERR_INVALID_ARG;
    const void *tok[] = {q, k, v, out, dout, dq, dk, dv};
    for (const void *t : tok)
        if (!aligned16(t)) return EVO_ERR_ALIGNMENT;
    if ((gate && !aligned16(gate)) || (dgate && !aligned16(dgate)) || (bias && !aligned16(bias)) ||
        (dbias && !aligned16(dbias)) || !aligned4(lse))
        return EVO_ERR_ALIGNMENT;
    return EVO_OK;
}

int bwd_impl(const evo_attn_dims *dims, const void *q, const void *k, const void *v, const void *gate,
             const void *bias, const uint8_t *key_mask, const void *out, const float *lse, const void *dout,
             void *dq, void *dk, void *dv, void *dgate, float *dbias, void *workspace, size_t workspace_bytes,
             void *stream, evo::Tracer *tr) {
    evo::Problem p;
    int st = check_bwd_args(dims, q, k, v, gate, bias, out, lse, dout, dq, dk, dv, dgate, dbias, &p);
    if (st) return st;
    if (p.N == 0 || p.L == 0) return EVO_OK;  // nothing is read or written
    const evo::BwdPlan plan = evo::plan_bwd(p, bias != nullptr);
    if (!workspace || workspace_bytes < plan.total || ((uintptr_t)workspace & 255u) != 0) return EVO_ERR_WORKSPACE;
    if (tr && tr->n < evo::bwd_kernel_count(bias != nullptr) + 1) return EVO_ERR_INVALID_ARG;
    if (tr)
        for (int i = 0; i < tr->n; ++i)
            if (!tr->ev[i]) return EVO_ERR_INVALID_ARG;
    evo::BwdPtrs x{q, k, v, gate, bias, key_mask, out, lse, dout, dq, dk, dv, dgate, dbias};
    hipError_t e = evo::launch_bwd(p, x, workspace, plan, (hipStream_t)stream, tr);
    return e == hipSuccess ? EVO_OK : EVO_ERR_HIP;
}

}  // namespace

int evo_attn_bwd(const evo_attn_dims *dims, const void *q, const void *k, const void *v, const void *gate,
                 const void *bias, const uint8_t *key_mask, const void *out, const float *lse, const void *dout,
                 void *dq, void *dk, void *dv, void *dgate, float *dbias, void *workspace, size_t workspace_bytes,
                 void *stream) {
    return bwd_impl(dims, q, k, v, gate, bias, key_mask, out, lse, dout, dq, dk, dv, dgate, dbias, workspace,
                    workspace_bytes, stream, nullptr);
}

int evo_attn_bwd_noalloc(const evo_attn_dims *dims, const void *q, const void *k, const void *v,
                         const void *gate, const void *bias, const uint8_t *key_mask, const void *out,
                         const float *lse, const void *dout, void *dq, void *dk, void *dv, void *dgate,
                         float *dbias, void *stream) {
    evo::Problem p;
    int st = check_bwd_args(dims, q, k, v, gate, bias, out, lse, dout, dq, dk, dv, dgate, dbias, &p);
    if (st) return st;
    if (p.N == 0 || p.L == 0) return EVO_OK;  // nothing is read or written
    // the plan takes fewer dBias row chunks where that brings it under the
    // buffer; a problem that does not fit even then is refused here, before
    // any HIP call
    const evo::BwdPlan plan = evo::plan_bwd(p, bias != nullptr, evo::kNoAllocScratchBytes);
    if (plan.total > evo::kNoAllocScratchBytes) return EVO_ERR_SCRATCH_LIMIT;
    void *scratch = nullptr;
    if (evo::noalloc_scratch_ptr(&scratch) != hipSuccess) return EVO_ERR_HIP;
    evo::BwdPtrs x{q, k, v, gate, bias, key_mask, out, lse, dout, dq, dk, dv, dgate, dbias};
    hipError_t e = evo::launch_bwd(p, x, scratch, plan, (hipStream_t)stream, nullptr);
    return e == hipSuccess ? EVO_OK : EVO_ERR_HIP;
}

size_t evo_attn_bwd_noalloc_scratch_bytes(void) { return evo::kNoAllocScratchBytes; }

int evo_attn_bwd_kernel_count(int has_bias) { return evo::bwd_kernel_count(has_bias != 0); }

int evo_attn_bwd_traced(const evo_attn_dims *dims, const void *q, const void *k, const void *v, const void *gate,
                        const void *bias, const uint8_t *key_mask, const void *out, const float *lse,
                        const void *dout, void *dq, void *dk, void *dv, void *dgate, float *dbias, void *workspace,
                        size_t workspace_bytes, void *const *events, int n_events, void *stream) {
    if (!events || n_events < 1) return EVO_ERR_INVALID_ARG;
    evo::Tracer tr;
    tr.ev = (hipEvent_t const *)events;
    tr.n = n_events;
    return bwd_impl(dims, q, k, v, gate, bias, key_mask, out, lse, dout, dq, dk, dv, dgate, dbias, workspace,
                    workspace_bytes, stream, &tr);
}

}  // extern "C"
