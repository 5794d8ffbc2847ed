/*
 * evo_attn.h -- C ABI of the MI355X (gfx950) Evoformer attention library.
 *
 * The library computes the gated multi-head attention with pair bias that
 * every Evoformer attention module runs (MSA row attention with pair bias,
 * MSA column attention, extra-MSA row attention, triangle attention around
 * the starting and the ending node), forward and backward:
 *
 *     o = sigmoid(g) * softmax(Q K^T / sqrt(d) + mask_bias + pair_bias) V
 *
 * ScaleFold (arXiv 2404.11068), Section 3.3, "Multi Head Attention": the
 * pair-bias term is added to the logits before the softmax, which rules out a
 * stock FlashAttention kernel; the paper fuses all of MHA into one
 * FlashAttention-style kernel.  Section 2.1 lists the four Evoformer modules
 * that contain this attention.  The exact semantics implemented here:
 *
 *   for row r (bias plane b = r / rows_per_bias), head h, query i, key j:
 *     s[i][j] = (1/sqrt(d)) sum_c Q[r,i,h,c] K[r,j,h,c] + bias[b,h,i,j]
 *     keys with key_mask[r,j] == 0 are excluded from the softmax
 *     P       = softmax_j(s),  A[i] = sum_j P[i][j] V[r,j,h,:]
 *     O       = sigmoid(G) * A         (no gate: O = A)
 *     lse[r,h,i] = log(sum_{kept j} exp(s[i][j]))      (natural log, fp32)
 *   A query whose keys are all masked gets O = 0, lse = -inf, zero gradients.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All tensor pointers are DEVICE pointers owned by the caller.  The library
 *   never allocates, frees or synchronises device memory; every call only
 *   enqueues kernels on `stream` (a hipStream_t; NULL = the null stream), so
 *   calls may be captured into a HIP graph.  Calls return as soon as the work
 *   is enqueued.
 * - Process-wide state, all of it set once: the environment variable
 *   EVO_ATTN_QBIAS_WAVES (a positive integer; default 4096) is read on the
 *   first backward plan of the process and fixes, for the rest of the
 *   process, how many waves the two-pass backward's dQ/dBias pass aims for
 *   (and so its row chunks and workspace size: set it before the first
 *   call, since evo_attn_bwd_workspace_size and evo_attn_bwd must see the
 *   same value); and the fixed scratch of evo_attn_bwd_noalloc (below), with
 *   its per-device address, looked up on the first such call on a device.
 *   One more environment variable is read on every evo_attn_fwd call and
 *   kept nowhere: EVO_ATTN_FWD_ROWS=0 selects the one-(row, head)-per-
 *   workgroup forward where the row-walking one (bias rows held in registers
 *   across the rows of one head) would run; both give the same bits.
 * - Token tensors Q, K, V, G, O, dO, dQ, dK, dV, dG share one layout: element
 *   (r, t, h, c) lives at  base + r*stride_row + t*stride_tok + h*head_dim + c
 *   (strides in ELEMENTS; the [H, d] block of a token is contiguous).  The
 *   contiguous [N, L, H, d] layout has stride_row = L*H*d, stride_tok = H*d.
 *   A transposed view (stride_row = H*d, stride_tok = L*H*d over an
 *   [L, L, H, d] pair representation) gives triangle attention around the
 *   ending node without a copy.
 * - bias (if given) is contiguous [B, H, L, L] in the working dtype with
 *   B = n_rows / rows_per_bias; dbias is contiguous [B, H, L, L] fp32.
 * - key_mask (if given) is contiguous [N, L] bytes, nonzero = keep.
 * - lse is contiguous [N, H, L] fp32.
 * - Outputs are overwritten, never accumulated into.
 * - Every argument is validated on the host before any HIP call; an invalid
 *   call enqueues nothing and returns a nonzero status.  Nothing is printed,
 *   thrown or aborted.  Non-finite input values are not checked.
 */
#ifndef EVO_ATTN_H
#define EVO_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* working dtype of Q, K, V, G, O, bias, dO, dQ, dK, dV, dG */
enum evo_attn_dtype {
    EVO_DTYPE_F32 = 0,  /* IEEE fp32 throughout (fp32 MFMA) */
    EVO_DTYPE_BF16 = 1  /* bf16 storage and MFMA inputs, fp32 accumulation */
};

enum evo_attn_status {
    EVO_OK = 0,
    EVO_ERR_INVALID_ARG = 1, /* null required pointer, negative size, bad rows_per_bias or strides */
    EVO_ERR_UNSUPPORTED = 2, /* dtype, head_dim or seq_len outside the compiled set */
    EVO_ERR_ALIGNMENT = 3,   /* token pointers/strides must allow 16-byte vector access */
    EVO_ERR_WORKSPACE = 4,   /* workspace missing or smaller than evo_attn_bwd_workspace_size */
    EVO_ERR_HIP = 5,         /* a kernel launch failed (hipGetLastError after the launch) */
    EVO_ERR_SCRATCH_LIMIT = 6 /* evo_attn_bwd_noalloc: the problem needs more scratch than
                                 EVO_ATTN_NOALLOC_SCRATCH_BYTES */
};

/* Compiled limits: head_dim in {8, 16, 32, 64}; 0 <= seq_len <= EVO_ATTN_MAX_SEQ_LEN
 * (512) for bf16 with head_dim <= 32; seq_len <= EVO_ATTN_MAX_SEQ_LEN_WIDE (256)
 * for fp32 and for head_dim 64; fp32 with head_dim 64: seq_len <=
 * EVO_ATTN_MAX_SEQ_LEN_F32_D64 (128).  Each bound is the most keys whose
 * staged tiles the kernels hold in a workgroup's LDS (a row of 257..512 keys
 * runs as 16-wave workgroups).  Head dims 8, 16 and 32 cover every Evoformer
 * attention (MSA row and column, triangle, extra-MSA); head_dim 64 runs each
 * (row, head) as two workgroups that form the same logits from all 64 channels
 * and produce 32 output channels each.
 *
 * Accuracy limit of the bf16 backward: it forms D_i = sum_c dO_ic O_ic from the
 * saved bf16 output O, so D carries about 2^-9 * ||dO_i * O_i||_2 of rounding
 * (grows as sqrt(head_dim) for unit-size entries), and dS = P (dP - D) inherits
 * it in full where the softmax puts its mass on a single key.  At head_dim <= 32
 * the gradients stay within 2e-2 abs + 2e-2 rel of the exact ones on such
 * inputs; at head_dim 64 a strongly peaked softmax (logit gaps of tens) can put
 * single dBias elements a few percent past that bound.  dBias sums these terms
 * over the rows_per_bias rows of its plane: near-cancelling elements then keep
 * an absolute error that grows as sqrt(rows_per_bias) while the normwise error
 * does not (about 2e-3 of ||dBias||_2 at any row count).  With unit-size
 * random inputs single elements stay within the bound up to 256 rows per plane
 * at head_dim 32 and 2048 at head_dim 8, and were seen up to 1.6x / 3.2x past
 * it at 512 / 1024 rows per plane at head_dim 32. */
#define EVO_ATTN_MAX_SEQ_LEN 512
#define EVO_ATTN_MAX_SEQ_LEN_WIDE 256     /* fp32, or head_dim 64 */
#define EVO_ATTN_MAX_SEQ_LEN_F32_D64 128

typedef struct evo_attn_dims {
    int32_t dtype;         /* enum evo_attn_dtype */
    int32_t n_heads;       /* H >= 1 */
    int32_t head_dim;      /* d */
    int32_t reserved;      /* must be 0 */
    int64_t n_rows;        /* N >= 0: independent attention rows (batch x rows) */
    int64_t seq_len;       /* L >= 0: queries == keys */
    int64_t rows_per_bias; /* >= 1; N % rows_per_bias == 0; ignored when bias is NULL */
    int64_t stride_row;    /* elements between rows r and r+1 of every token tensor */
    int64_t stride_tok;    /* elements between tokens t and t+1; >= H*d;
                              seq_len * stride_tok * element size must stay
                              below 2^31 bytes (else EVO_ERR_UNSUPPORTED) */
} evo_attn_dims;

/*
 * Forward pass.
 *   q, k, v : required token tensors (input)
 *   gate    : gate logits (token tensor) or NULL for no gating
 *   bias    : pair bias [B,H,L,L] or NULL
 *   key_mask: [N,L] bytes or NULL (all keys kept)
 *   out     : O (token tensor, output; must not alias an input)
 *   lse     : [N,H,L] fp32 output, natural-log log-sum-exp of each query's
 *             logits; required (the backward consumes it)
 * Returns EVO_OK or an evo_attn_status.  An empty problem (N == 0 or L == 0)
 * validates dims and returns EVO_OK without launching anything or looking at
 * any pointer (which may then be NULL); the same holds for evo_attn_bwd.
 */
int evo_attn_fwd(const evo_attn_dims *dims, const void *q, const void *k, const void *v,
                 const void *gate, const void *bias, const uint8_t *key_mask, void *out,
                 float *lse, void *stream);

/*
 * Bytes of device workspace evo_attn_bwd needs for these dims (0 if dims is
 * invalid).  The value depends on the dims only; it may change between
 * library versions, so query it rather than hard-coding it.
 */
size_t evo_attn_bwd_workspace_size(const evo_attn_dims *dims);

/*
 * Backward pass (recomputes the softmax from the saved lse).
 *   q, k, v, gate, bias, key_mask : as passed to evo_attn_fwd
 *   out, lse : the forward's outputs
 *   dout     : dL/dO (token tensor)
 *   dq, dk, dv : gradient outputs (token tensors)
 *   dgate    : dL/dG output; NULL if and only if gate is NULL
 *   dbias    : dL/dbias [B,H,L,L] fp32 output (summed over the rows sharing
 *              each plane); NULL if and only if bias is NULL
 *   workspace, workspace_bytes : caller-owned device scratch of at least
 *              evo_attn_bwd_workspace_size(dims) bytes, 256-byte aligned;
 *              its contents on entry do not matter
 * Every sum (over keys, queries and the rows of a bias plane) runs in a
 * fixed order without atomics, so repeated calls give bitwise identical
 * results.
 */
int evo_attn_bwd(const evo_attn_dims *dims, const void *q, const void *k, const void *v,
                 const void *gate, const void *bias, const uint8_t *key_mask, const void *out,
                 const float *lse, const void *dout, void *dq, void *dk, void *dv, void *dgate,
                 float *dbias, void *workspace, size_t workspace_bytes, void *stream);

/*
 * Profiling variant of evo_attn_bwd (identical arguments and results).  The
 * caller passes n_events hipEvent_t handles it created; the library records
 * events[0] on `stream` before its first kernel and events[i] right after its
 * i-th kernel, so event pairs bracket single kernels.  Kernel order in this
 * version: [pair-bias transpose], dK/dV pass, dQ/dBias pass, [dBias reduce]
 * (bracketed entries only when bias != NULL).  The transpose runs only for
 * fp32 or a seq_len that is not a multiple of 8; otherwise the dK/dV pass reads
 * the bias as it is and events[0] and events[1] bracket no kernel (the slot is
 * kept so that the event count depends on has_bias alone).  n_events must be at least
 * evo_attn_bwd_kernel_count(bias != NULL) + 1 and every handle non-NULL,
 * else EVO_ERR_INVALID_ARG.  Meant for benchmarks; recording events costs a
 * few microseconds per call.
 */
int evo_attn_bwd_traced(const evo_attn_dims *dims, const void *q, const void *k, const void *v,
                        const void *gate, const void *bias, const uint8_t *key_mask,
                        const void *out, const float *lse, const void *dout, void *dq, void *dk,
                        void *dv, void *dgate, float *dbias, void *workspace,
                        size_t workspace_bytes, void *const *events, int n_events, void *stream);

/*
 * Backward pass that allocates nothing, for callers that cannot allocate
 * device memory or pass a workspace: code being captured into a HIP graph,
 * tight serving loops, harnesses that forbid hipMalloc.
 *
 * Same arguments and results as evo_attn_bwd without the workspace: the
 * scratch lives in a fixed buffer of EVO_ATTN_NOALLOC_SCRATCH_BYTES that the
 * library holds on every device it runs on, from the first call on that
 * device until the process ends.  The stream must belong to the current
 * device (the buffer is looked up for it on the first call there).
 *   - Calls on one device share that buffer: two calls that overlap in time
 *     on one device (different streams, or different host threads without
 *     ordering between their streams) race and give undefined results.
 *     Calls ordered on one stream are safe.  The buffer keeps the last
 *     call's contents; nothing in it needs clearing between calls.
 *   - A problem whose scratch does not fit is refused before any HIP call
 *     with EVO_ERR_SCRATCH_LIMIT.  Where fewer dBias partial planes make it
 *     fit, the call uses fewer (so its dBias may differ from evo_attn_bwd's
 *     in the order of the row sums, within rounding); otherwise results are
 *     bitwise those of evo_attn_bwd.
 *   - No hipMalloc, hipFree or other allocating call is made.
 */
#define EVO_ATTN_NOALLOC_SCRATCH_BYTES (64u << 20)
int evo_attn_bwd_noalloc(const evo_attn_dims *dims, const void *q, const void *k, const void *v,
                         const void *gate, const void *bias, const uint8_t *key_mask,
                         const void *out, const float *lse, const void *dout, void *dq, void *dk,
                         void *dv, void *dgate, float *dbias, void *stream);

/* EVO_ATTN_NOALLOC_SCRATCH_BYTES as compiled into the library. */
size_t evo_attn_bwd_noalloc_scratch_bytes(void);

/* Number of kernels one evo_attn_bwd call launches (has_bias: bias != NULL). */
int evo_attn_bwd_kernel_count(int has_bias);

/* Static, human-readable text for a status code (never NULL). */
const char *evo_attn_strerror(int status);

/* Library ABI version (major * 10000 + minor * 100 + patch). */
int evo_attn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* EVO_ATTN_H */
