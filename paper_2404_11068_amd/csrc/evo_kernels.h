// evo_kernels.h -- internal launch interface between the C ABI layer and the
// HIP kernels (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace evo {

struct Problem {
    int dtype;          // 0 = fp32, 1 = bf16
    int H, D;
    int64_t N, L, rpb;  // rpb: rows per bias plane
    int64_t srow, stok; // token-tensor strides, elements
};

struct FwdPtrs {
    const void *q, *k, *v, *g, *bias;
    const uint8_t *mask;
    void *out;
    float *lse;
};

struct BwdPtrs {
    const void *q, *k, *v, *g, *bias;
    const uint8_t *mask;
    const void *out;
    const float *lse;
    const void *dout;
    void *dq, *dk, *dv, *dg;
    float *dbias;
};

// Backward scratch plan: which kernels run and where each buffer lives
// inside the workspace.
//   fused (bf16, head_dim <= 32): one pass; the workspace holds only the
//     partial dBias planes (chunks > 1), at offset 0
//   otherwise: the dK/dV pass and the dQ/dBias pass, with dA, Dsum, the
//     transposed bias and the partial dBias planes in the workspace
struct BwdPlan {
    bool fused;
    int64_t chunks;          // row chunks per bias plane (dBias partial planes per plane and head)
    int64_t rows_per_chunk;  // rows handled by one workgroup of the dBias-producing pass
    int64_t n_wg;            // workgroups of the qbias kernel (two-pass plan)
    size_t off_da, off_dsum, off_biast, off_part, total;
};

// cap: largest workspace the caller can give; the plan takes fewer row chunks
// (fewer partial dBias planes) to stay under it where it can (callers check
// .total against the cap)
BwdPlan plan_bwd(const Problem &p, bool has_bias, size_t cap = ~(size_t)0);

// Fixed device scratch of the no-alloc backward (EVO_ATTN_NOALLOC_SCRATCH_BYTES
// per device): its device address on the current device, looked up on the
// first call per device.
constexpr size_t kNoAllocScratchBytes = (size_t)64 << 20;
hipError_t noalloc_scratch_ptr(void **out);

// Optional stage markers: records caller-owned events on the launch stream
// before the first kernel and after each kernel (profiling only).
struct Tracer {
    hipEvent_t const *ev = nullptr;
    int n = 0, next = 0;
    void mark(hipStream_t s) {
        if (ev && next < n) (void)hipEventRecord(ev[next], s);
        ++next;
    }
    // record the events no kernel claimed (they bracket nothing)
    void fill(hipStream_t s) {
        while (ev && next < n) mark(s);
    }
};

// single-pass backward (evo_bwd_fused.hip)
bool fused_bwd_supported(const Problem &p, bool has_bias);
void fused_bwd_chunks(const Problem &p, bool has_bias, int64_t *chunks, int64_t *rows_per_chunk);
size_t fused_bwd_partial_bytes(const Problem &p, int64_t chunks);
hipError_t launch_bwd_fused(const Problem &p, const BwdPtrs &x, void *ws, int64_t chunks, int64_t rows_per_chunk,
                            hipStream_t s, Tracer &tr);

// kernels launched by one backward call (for Tracer sizing)
int bwd_kernel_count(bool has_bias);

hipError_t launch_fwd(const Problem &p, const FwdPtrs &x, hipStream_t s);
hipError_t launch_bwd(const Problem &p, const BwdPtrs &x, void *ws, const BwdPlan &plan,
                      hipStream_t s, Tracer *tr = nullptr);

// LayerNorm over the last axis of a contiguous [R, C] tensor
struct LnProblem {
    int dtype;   // 0 = fp32, 1 = bf16 (x, y, dy, dx); parameters and statistics are fp32
    int C;
    int64_t R;
    float eps;
};

struct LnPtrs {
    const void *x;
    const float *w, *b;
    void *y;
    float *mean, *rstd;  // nullable
};

struct LnBwdPtrs {
    const void *x;
    const float *w, *mean, *rstd;
    const void *dy;
    void *dx;
    float *dw, *db;
};

bool ln_supported_cols(int C);
size_t ln_bwd_workspace(const LnProblem &p);
hipError_t launch_ln_fwd(const LnProblem &p, const LnPtrs &x, hipStream_t s);
hipError_t launch_ln_bwd(const LnProblem &p, const LnBwdPtrs &x, void *ws, hipStream_t s, Tracer *tr = nullptr);

// LayerNorm + P batched projections (bf16): out_p = LN(x) W_p^T + b_p
struct PjArgs {
    const void *x;            // [R, C] bf16
    const float *lnw, *lnb;   // [C], or both null for a plain linear layer
    const void *W;            // [P*HD, C] bf16
    const float *bias;        // [P*HD] or null
    void *out0, *out1, *out2, *out3;  // [R, HD] bf16 each (first P used)
    float *mean, *rstd;       // [R] or null (both or neither)
    void *y;                  // [R, C] bf16 normalised input (saved for the backward) or null
    int64_t R;
    int C, HD, P;
    float eps;
};

// backward of the fused LayerNorm + projections
struct PjBwdArgs {
    const void *x;            // [R, C] bf16
    const float *lnw;         // [C], or null for a plain linear layer
    const float *mean, *rstd; // [R]
    const void *y;            // [R, C] bf16 normalised input from the forward (x without LayerNorm)
    const void *W;            // [P*HD, C] bf16
    const void *dout0, *dout1, *dout2, *dout3;  // [R, HD] bf16
    void *dx;                 // [R, C] bf16
    float *dW;                // [P*HD, C]
    float *dbias;             // [P*HD] or null
    float *dlnw, *dlnb;       // [C]
    int64_t R;
    int C, HD, P;
};

struct PjBwdPlan {
    int64_t n_chunks, chunk_tokens;   // token chunks of the weight-gradient pass
    size_t off_dy, off_ln, off_dw, off_db, total;
};

// ln == false: a plain linear layer (no LayerNorm; lnw, mean, rstd, dlnw,
// dlnb null and y = x), dY written straight to dx
PjBwdPlan plan_proj_bwd(int64_t R, int C, int HD, int P, bool ln = true);
hipError_t launch_ln_proj_bwd(const PjBwdArgs &a, void *ws, const PjBwdPlan &plan, hipStream_t s);

// LayerNorm of pair entries projected to per-head logit biases (bf16)
struct PbArgs {
    const void *z;            // [B, Li, Lj, C] bf16
    const float *lnw, *lnb;   // [C]
    const void *W;            // [H, C] bf16
    void *out;                // [B, H, Li, Lj] (or [B, H, Lj, Li] when transpose) bf16
    float *mean, *rstd;       // [B, Li, Lj] or null (both or neither)
    int64_t B;
    int Li, Lj, C, H, transpose;
    float eps;
};

bool pair_bias_supported(int C, int H);
hipError_t launch_pair_bias(const PbArgs &a, hipStream_t s);

// backward of the pair bias: dz, dW [H, C], dln_w, dln_b from dbias (fp32,
// the forward's output layout)
struct PbBwdArgs {
    const void *z;            // [B, Li, Lj, C] bf16
    const float *lnw, *lnb;   // [C]
    const void *W;            // [H, C] bf16
    const float *dbias;       // [B, H, Li, Lj] (or [B, H, Lj, Li] when transpose) fp32
    void *dz;                 // [B, Li, Lj, C] bf16
    float *dW, *dlnw, *dlnb;  // [H, C], [C], [C]
    int64_t B;
    int Li, Lj, C, H, transpose;
    float eps;
};

bool pair_bias_bwd_supported(int C, int H);
int64_t pair_bias_bwd_workgroups(int64_t B, int Li, int Lj, int C);
size_t pair_bias_bwd_workspace(int64_t B, int Li, int Lj, int C, int H);
hipError_t launch_pair_bias_bwd(const PbBwdArgs &a, void *ws, hipStream_t s);

bool proj_supported(int C, int HD, int P);
hipError_t launch_ln_proj(const PjArgs &a, hipStream_t s);

}  // namespace evo

// fused optimizer step (types from include/evo_optim.h)
struct evo_mt_tensor;
struct evo_mt_chunk;
struct evo_adam_swa_hparams;
namespace evo {
hipError_t launch_adam_swa(const evo_adam_swa_hparams &hp, const evo_mt_tensor *tensors, int32_t n_tensors,
                           const evo_mt_chunk *chunks, int32_t n_chunks, const float *grad_scale, hipStream_t s);
hipError_t launch_clip_scale(const evo_mt_tensor *tensors, int32_t n_tensors, const evo_mt_chunk *chunks,
                             int32_t n_chunks, float max_norm, float *ws, float *norm_out, float *scale_out,
                             hipStream_t s);
}  // namespace evo
