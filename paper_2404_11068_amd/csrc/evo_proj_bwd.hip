// evo_proj_bwd.hip -- backward of the fused LayerNorm + batched projections,
// gfx950.
//
// With y = LN(x) (saved by the forward as bf16) and upstream gradients
// dout_p of the P projections:
//
//   dY      = sum_p dout_p W_p          [R, C]   (dy_kernel, MFMA)
//   dx, dln = LayerNorm backward of dY           (the LayerNorm kernels)
//   dW_p    = dout_p^T y                [HD, C]  (dw_kernel, MFMA, per token chunk)
//   dbias_p = sum over tokens of dout_p          (same kernel, a ones operand)
//
// followed by a fixed-order sum of the per-chunk dW / dbias partials.  In
// both products the contraction runs along an axis that is not contiguous in
// one operand (features of W in dY, tokens in dW), so those operands are
// staged in LDS and read with the transposing LDS read (ds_read_b64_tr_b16),
// which yields the MFMA fragment directly.  dY is rounded to bf16 (the
// gradient precision between the layers) before the LayerNorm backward.
#include <stdlib.h>

#include "evo_frag.h"
#include "evo_kernels.h"

namespace evo {
namespace {

constexpr int kPbwWaves = 8;

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// features per workgroup of the weight-gradient pass: a block never spans two
// projections (it divides HD); 128 when the channel tiles alone would leave
// waves idle (C = 64)
inline int proj_bwd_fb(int C, int HD) {
    if (C == 64 && HD % 128 == 0) return 128;
    return HD % 64 == 0 ? 64 : 32;
}

__device__ __forceinline__ const void *dout_ptr(const PjBwdArgs &a, int p) {
    return p == 0 ? a.dout0 : p == 1 ? a.dout1 : p == 2 ? a.dout2 : a.dout3;
}

// ---------------------------------------------------------------------------
// dY tile of 128 tokens x C channels.  Output tiles (token block tb, channel
// tile ct): wave w takes tb = w % 4 and channel tiles ct = w / 4 + 2 j.  The
// weight streams through LDS in chunks of 32 feature rows (double-buffered,
// the next chunk's global loads issued before this chunk's products).
template <int C>
__global__ __launch_bounds__(64 * kPbwWaves) void dy_kernel(PjBwdArgs a, void *__restrict__ dy) {
    constexpr int TM = 128;
    constexpr int NCT = C / 32;               // channel tiles
    constexpr int TPW = NCT / 2 > 0 ? NCT / 2 : 1;  // channel tiles per wave (C >= 64)
    constexpr int WSTR = C + 8;               // LDS row stride of a weight chunk (elements)
    constexpr int NWL = (32 * C / 8 + 64 * kPbwWaves - 1) / (64 * kPbwWaves);  // 16-byte loads per thread
    constexpr int OSTR = 40;                  // staging row stride (elements) of a 32x32 output tile
    __shared__ __attribute__((aligned(16))) uint16_t wl[2][32 * WSTR];
    __shared__ __attribute__((aligned(16))) uint16_t stage[kPbwWaves][32 * OSTR];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 31, h = lane >> 5;
    const int tb = wave & 3, cg = wave >> 2;
    const int64_t row0 = (int64_t)blockIdx.x * TM;
    int64_t nrows = a.R - row0;
    nrows = nrows < TM ? nrows : TM;
    const int NFC = a.P * a.HD / 32;
    const rsrc_t rW = make_buf(a.W, (uint32_t)(a.P * a.HD) * C * 2u);

    u32x4 wr[NWL];
    auto load_w = [&](int fc) {
#pragma unroll
        for (int j = 0; j < NWL; ++j) {
            const int idx = tid + j * 64 * kPbwWaves;
            const int r = idx / (C / 8), c8 = idx % (C / 8);
            wr[j] = bload16(rW, idx < 32 * C / 8 ? (uint32_t)((fc * 32 + r) * C + c8 * 8) * 2u : kOOB);
        }
    };
    auto store_w = [&](int buf) {
#pragma unroll
        for (int j = 0; j < NWL; ++j) {
            const int idx = tid + j * 64 * kPbwWaves;
            if (idx < 32 * C / 8) {
                const int r = idx / (C / 8), c8 = idx % (C / 8);
                *(u32x4 *)&wl[buf][r * WSTR + c8 * 8] = wr[j];
            }
        }
    };

    f32x16 acc[TPW];
#pragma unroll
    for (int j = 0; j < TPW; ++j) acc[j] = zero16();
    load_w(0);
    store_w(0);
    __syncthreads();
    for (int fc = 0; fc < NFC; ++fc) {
        if (fc + 1 < NFC) load_w(fc + 1);
        // A: dout rows of this token block, the chunk's 32 features (k32 order)
        const int p = (fc * 32) / a.HD, fl = (fc * 32) % a.HD;
        const rsrc_t ro = make_buf((const char *)dout_ptr(a, p) + row0 * a.HD * 2, (uint32_t)nrows * a.HD * 2u);
        const uint32_t rb = (uint32_t)((tb * 32 + n) * a.HD + fl) * 2u;
        Tr<bf16_t>::K32 af;
        af.v[0] = __builtin_bit_cast(bf16x8, bload16(ro, rb + 16u * h));
        af.v[1] = __builtin_bit_cast(bf16x8, bload16(ro, rb + 32u + 16u * h));
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
            const int ct = cg + 2 * j;
            if (ct < NCT) {
                const Tr<bf16_t>::K32 bf = load_k32_tr(&wl[fc & 1][ct * 32], WSTR, 0, 32, lane);
                Tr<bf16_t>::mma_k32(acc[j], af, bf);
            }
        }
        if (fc + 1 < NFC) store_w((fc + 1) & 1);
        __syncthreads();
    }

    // epilogue: D[token rho(i,h)][channel ct*32 + sig(n)] -> bf16 -> token rows
    const rsrc_t rd = make_buf((char *)dy + row0 * C * 2, (uint32_t)nrows * C * 2);
    uint16_t *st = stage[wave];
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
        const int ct = cg + 2 * j;
        if (ct >= NCT) continue;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int t = 8 * (i / 4) + 4 * h + (i % 4);
            st[t * OSTR + sig(n)] = __builtin_bit_cast(uint16_t, (__bf16)acc[j][i]);
        }
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int t = q * 16 + (lane >> 2), c4 = lane & 3;
            const u32x4 v = *(const u32x4 *)&st[t * OSTR + c4 * 8];
            bstore16(v, rd, (uint32_t)((tb * 32 + t) * C + ct * 32 + c4 * 8) * 2u);
        }
        __builtin_amdgcn_wave_barrier();
    }
}

// ---------------------------------------------------------------------------
// Partial dW (FB features x C channels) and dbias over one chunk of tokens.
// Tokens go through LDS 32 at a time (dout [32][FB] and y [32][C] rows,
// double-buffered through registers); wave w owns output tiles
// (feature tile, channel tile) = w, w + 8, ... of the (FB/32) x (C/32) grid.
template <int C, int FB>
__global__ __launch_bounds__(64 * kPbwWaves) void dw_kernel(PjBwdArgs a, int64_t chunk_tokens,
                                                          float *__restrict__ part_w, float *__restrict__ part_b) {
    constexpr int NFT = FB / 32, NCT = C / 32, NT = NFT * NCT;
    constexpr int TPW = (NT + kPbwWaves - 1) / kPbwWaves;
    constexpr int DSTR = FB + 8, YSTR = C + 8;
    constexpr int ND = (32 * FB / 8 + 64 * kPbwWaves - 1) / (64 * kPbwWaves);
    constexpr int NY = (32 * C / 8 + 64 * kPbwWaves - 1) / (64 * kPbwWaves);
    __shared__ __attribute__((aligned(16))) uint16_t dl[2][32 * DSTR];
    __shared__ __attribute__((aligned(16))) uint16_t yl[2][32 * YSTR];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 31, h = lane >> 5;
    const int F = a.P * a.HD;
    const int fb = blockIdx.x;               // feature block
    const int64_t chunk = blockIdx.y;
    const int64_t t_begin = chunk * chunk_tokens;
    int64_t t_end = t_begin + chunk_tokens;
    t_end = t_end < a.R ? t_end : a.R;
    const int f0 = fb * FB;
    // the feature block lies inside one projection (HD is a multiple of FB)
    const int p = f0 / a.HD, fl0 = f0 % a.HD;

    u32x4 dr[ND], yr[NY];
    auto load_sub = [&](int64_t t0) {
        // dout rows t0..t0+31 of this projection's features fl0..fl0+FB
        const int64_t nt = t_end - t0 < 32 ? t_end - t0 : 32;
        const rsrc_t rd_ = make_buf((const char *)dout_ptr(a, p) + t0 * a.HD * 2, nt > 0 ? (uint32_t)nt * a.HD * 2u : 0u);
        const rsrc_t ry_ = make_buf((const char *)a.y + t0 * C * 2, nt > 0 ? (uint32_t)nt * C * 2u : 0u);
#pragma unroll
        for (int j = 0; j < ND; ++j) {
            const int idx = tid + j * 64 * kPbwWaves;
            const int r = idx / (FB / 8), c8 = idx % (FB / 8);
            dr[j] = bload16(rd_, idx < 32 * FB / 8 ? (uint32_t)(r * a.HD + fl0 + c8 * 8) * 2u : kOOB);
        }
#pragma unroll
        for (int j = 0; j < NY; ++j) {
            const int idx = tid + j * 64 * kPbwWaves;
            const int r = idx / (C / 8), c8 = idx % (C / 8);
            yr[j] = bload16(ry_, idx < 32 * C / 8 ? (uint32_t)(r * C + c8 * 8) * 2u : kOOB);
        }
    };
    auto store_sub = [&](int buf) {
#pragma unroll
        for (int j = 0; j < ND; ++j) {
            const int idx = tid + j * 64 * kPbwWaves;
            if (idx < 32 * FB / 8) {
                const int r = idx / (FB / 8), c8 = idx % (FB / 8);
                *(u32x4 *)&dl[buf][r * DSTR + c8 * 8] = dr[j];
            }
        }
#pragma unroll
        for (int j = 0; j < NY; ++j) {
            const int idx = tid + j * 64 * kPbwWaves;
            if (idx < 32 * C / 8) {
                const int r = idx / (C / 8), c8 = idx % (C / 8);
                *(u32x4 *)&yl[buf][r * YSTR + c8 * 8] = yr[j];
            }
        }
    };

    // all-ones B operand: D[f][n] += sum over the tokens of dout[t][f]
    Tr<bf16_t>::K32 ones;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int s = 0; s < 8; ++s) ones.v[t][s] = (__bf16)1.0f;
    // the owner of (feature tile, channel tile 0) also sums dbias for that feature tile
    f32x16 acc[TPW], accb[TPW];
#pragma unroll
    for (int j = 0; j < TPW; ++j) acc[j] = accb[j] = zero16();

    const int64_t nsub = (t_end - t_begin + 31) / 32;
    load_sub(t_begin);
    store_sub(0);
    __syncthreads();
    for (int64_t sb = 0; sb < nsub; ++sb) {
        if (sb + 1 < nsub) load_sub(t_begin + (sb + 1) * 32);
        const int buf = (int)(sb & 1);
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
            const int tile = wave + j * kPbwWaves;
            if (tile < NT) {
                const int ft = tile / NCT, ct = tile % NCT;
                const Tr<bf16_t>::K32 af = load_k32_tr(&dl[buf][ft * 32], DSTR, 0, 32, lane);
                const Tr<bf16_t>::K32 bf = load_k32_tr(&yl[buf][ct * 32], YSTR, 0, 32, lane);
                Tr<bf16_t>::mma_k32(acc[j], af, bf);
                if (ct == 0) Tr<bf16_t>::mma_k32(accb[j], af, ones);
            }
        }
        if (sb + 1 < nsub) store_sub((sb + 1) & 1);
        __syncthreads();
    }

    // partial tiles: D[feature ft*32 + sig(rho(i,h))][channel ct*32 + sig(n)]
    const rsrc_t rpw = make_buf(part_w + chunk * (int64_t)F * C, (uint32_t)F * C * 4u);
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
        const int tile = wave + j * kPbwWaves;
        if (tile >= NT) continue;
        const int ft = tile / NCT, ct = tile % NCT;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int f = f0 + ft * 32 + sig(8 * (i / 4) + 4 * h + (i % 4));
            bstore4(__float_as_uint(acc[j][i]), rpw, (uint32_t)(f * C + ct * 32 + sig(n)) * 4u);
        }
    }
    if (part_b) {
        const rsrc_t rpb = make_buf(part_b + chunk * (int64_t)F, (uint32_t)F * 4u);
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
            const int tile = wave + j * kPbwWaves;
            if (tile >= NT || tile % NCT != 0) continue;
            const int ft = tile / NCT;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int f = f0 + ft * 32 + sig(8 * (i / 4) + 4 * h + (i % 4));
                bstore4(__float_as_uint(accb[j][i]), rpb, n == 0 ? (uint32_t)f * 4u : kOOB);
            }
        }
    }
}

// out[x] = sum_k part[k][x] in k order, four columns per thread
__global__ __launch_bounds__(256) void colsum_kernel(const float *__restrict__ part, int64_t n_part, int64_t width,
                                                    float *__restrict__ out) {
    const int64_t x4 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
    if (x4 >= width) return;
    const rsrc_t rp = make_buf(part, (uint32_t)(n_part * width * 4));
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
    int64_t k = 0;
    for (; k + 4 <= n_part; k += 4) {
        f32x4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = __builtin_bit_cast(f32x4, bload16(rp, (uint32_t)((k + u) * width + x4) * 4u));
#pragma unroll
        for (int u = 0; u < 4; ++u) s += v[u];
    }
    for (; k < n_part; ++k) s += __builtin_bit_cast(f32x4, bload16(rp, (uint32_t)(k * width + x4) * 4u));
    const rsrc_t ro = make_buf(out, (uint32_t)(width * 4));
    bstore16(__builtin_bit_cast(u32x4, s), ro, (uint32_t)x4 * 4u);
}

template <int C>
hipError_t launch_c(const PjBwdArgs &a, void *ws, const PjBwdPlan &plan, hipStream_t s) {
    char *w = (char *)ws;
    void *dy = w + plan.off_dy;
    const int64_t nt = (a.R + 127) / 128;
    hipLaunchKernelGGL((dy_kernel<C>), dim3((unsigned)nt), dim3(64 * kPbwWaves), 0, s, a, dy);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // LayerNorm backward of dY (bf16) -> dx, dln_w, dln_b
    LnProblem lp{1, C, a.R, 0.0f};
    LnBwdPtrs lx{a.x, a.lnw, a.mean, a.rstd, dy, a.dx, a.dlnw, a.dlnb};
    e = launch_ln_bwd(lp, lx, w + plan.off_ln, s);
    if (e != hipSuccess) return e;
    const int F = a.P * a.HD;
    float *pw = (float *)(w + plan.off_dw);
    float *pb = a.dbias ? (float *)(w + plan.off_db) : nullptr;
    const int fb = proj_bwd_fb(C, a.HD);
    const dim3 grid((unsigned)(F / fb), (unsigned)plan.n_chunks);
    if (fb == 128) {
        hipLaunchKernelGGL((dw_kernel<C, 128>), grid, dim3(64 * kPbwWaves), 0, s, a, plan.chunk_tokens, pw, pb);
    } else if (fb == 64) {
        hipLaunchKernelGGL((dw_kernel<C, 64>), grid, dim3(64 * kPbwWaves), 0, s, a, plan.chunk_tokens, pw, pb);
    } else {
        hipLaunchKernelGGL((dw_kernel<C, 32>), grid, dim3(64 * kPbwWaves), 0, s, a, plan.chunk_tokens, pw, pb);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t wdw = (int64_t)F * C;
    hipLaunchKernelGGL(colsum_kernel, dim3((unsigned)((wdw / 4 + 255) / 256)), dim3(256), 0, s, pw, plan.n_chunks,
                       wdw, a.dW);
    e = hipGetLastError();
    if (e != hipSuccess || !a.dbias) return e;
    hipLaunchKernelGGL(colsum_kernel, dim3((unsigned)((F / 4 + 255) / 256)), dim3(256), 0, s, pb, plan.n_chunks,
                       (int64_t)F, a.dbias);
    return hipGetLastError();
}

}  // namespace

PjBwdPlan plan_proj_bwd(int64_t R, int C, int HD, int P) {
    PjBwdPlan pl{};
    const int F = P * HD;
    const int FB = proj_bwd_fb(C, HD);
    const int64_t nfb = F / FB > 0 ? F / FB : 1;
    // enough (feature block, token chunk) workgroups to cover the CUs twice,
    // chunks of whole 32-token sub-blocks
    int64_t nch = (512 + nfb - 1) / nfb;
    const int64_t cap = ((int64_t)1 << 30) / ((int64_t)F * C * 4);  // partials below 1 GiB
    if (nch > cap) nch = cap > 0 ? cap : 1;
    const int64_t nsub = (R + 31) / 32;
    if (nch > nsub) nch = nsub > 0 ? nsub : 1;
    int64_t subs = (nsub + nch - 1) / nch;
    pl.chunk_tokens = subs * 32;
    pl.n_chunks = R > 0 ? (R + pl.chunk_tokens - 1) / pl.chunk_tokens : 1;
    LnProblem lp{1, C, R, 0.0f};
    size_t off = 0;
    pl.off_dy = off;
    off += align256((size_t)R * C * 2);
    pl.off_ln = off;
    off += align256(ln_bwd_workspace(lp));
    pl.off_dw = off;
    off += align256((size_t)pl.n_chunks * F * C * 4);
    pl.off_db = off;
    off += align256((size_t)pl.n_chunks * F * 4);
    pl.total = off;
    return pl;
}

hipError_t launch_ln_proj_bwd(const PjBwdArgs &a, void *ws, const PjBwdPlan &plan, hipStream_t s) {
    switch (a.C) {
        case 64: return launch_c<64>(a, ws, plan, s);
        case 128: return launch_c<128>(a, ws, plan, s);
        case 256: return launch_c<256>(a, ws, plan, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace evo
