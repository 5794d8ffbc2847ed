// evo_proj.hip -- fused LayerNorm + batched linear projections, gfx950.
//
// ScaleFold, Section 3.3: the four linear layers in front of each Evoformer
// attention (query, key, value, gate) read the same normalised input and do
// not depend on each other, so the paper batches them into one product and
// fuses LayerNorm, the four GEMMs and the attention.  Here one kernel does
// LayerNorm and the four projections and writes each result straight into
// the attention's token layout ([rows, H*d], i.e. [N, L, H, d]):
//
//   out_p[t, :] = LN(x[t, :]) @ W[p*HD : (p+1)*HD, :]^T + bias[p*HD : (p+1)*HD]
//
// Workgroup = 8 waves (two per SIMD) and a tile of TM = 32*TB tokens:
//   1. LayerNorm of the tile (rows spread over the waves, statistics in
//      registers as in the stand-alone LayerNorm kernel), rounded to bf16 into
//      LDS as [token][C] rows padded by 16 bytes (conflict-free 16-byte reads).
//   2. The P*HD output features split into 32-feature tiles; wave w takes
//      tiles w, w+8, ...  For a tile it holds the 32 weight rows (torch
//      Linear layout [features, C], so k is contiguous) as MFMA A fragments in
//      registers and runs
//      v_mfma_f32_32x32x16_bf16 against every token block of the LDS tile
//      (B fragments), TB independent accumulators.
//   3. D[feature][token] puts 4 consecutive features of one token in each
//      lane's register quads; the epilogue adds the bias, rounds to bf16,
//      turns the tile into token rows through a wave-private LDS staging
//      area and stores 16 bytes per lane, 64 contiguous bytes per token row.
// Tails: a buffer resource per output that ends at the last valid row drops
// the stores of padding tokens; their loads read zeros.
#include <stdlib.h>

#include "evo_frag.h"
#include "evo_kernels.h"

namespace evo {
namespace {

constexpr int kPjWaves = 8;

__device__ __forceinline__ void bstore8(u32x2 v, rsrc_t r, uint32_t off) {
    __builtin_amdgcn_raw_buffer_store_b64(v, r, off, 0, 0);
}

template <int LPR>
__device__ __forceinline__ float pj_row_sum(float v) {
    if constexpr (LPR >= 2) v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
    if constexpr (LPR >= 4) v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, false));
    if constexpr (LPR >= 8) v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x141, 0xF, 0xF, false));
    if constexpr (LPR >= 16) v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x140, 0xF, 0xF, false));
    if constexpr (LPR >= 32) v += __shfl_xor(v, 16, 64);
    return v;
}

template <int C, int TB>
struct PjGeom {
    static constexpr int TM = 32 * TB;              // tokens per workgroup
    static constexpr int LPR = C / 8;               // lanes per row in the LayerNorm
    static constexpr int RPW = 64 / LPR;            // rows per wave slot
    static constexpr int SLOTS = TM / kPjWaves / RPW;
    static constexpr int KS = C / 16;               // MFMA k-steps
    static constexpr int STRIDE = 2 * C + 16;       // LDS bytes per token row
    static constexpr int OSTRIDE = 80;              // staging bytes per token row (32 bf16 + pad)
    static constexpr int OBYTES = TM * OSTRIDE;     // staging bytes per wave
    static_assert(C % 16 == 0 && LPR <= 32 && SLOTS >= 1, "unsupported shape");
};

template <int C, int TB>
__global__ __launch_bounds__(64 * kPjWaves) void ln_proj_kernel(PjArgs a) {
    using G = PjGeom<C, TB>;
    __shared__ __attribute__((aligned(16))) char lds[G::TM * G::STRIDE + kPjWaves * G::OBYTES];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform: scalar addressing
    const int64_t row0 = (int64_t)blockIdx.x * G::TM;
    int64_t nrows = a.R - row0;
    nrows = nrows < G::TM ? nrows : G::TM;

    // ---- 1. LayerNorm of the tile into LDS ---------------------------------
    {
        const int li = lane % G::LPR, rs = lane / G::LPR;
        const rsrc_t rx = make_buf((const char *)a.x + row0 * C * 2, (uint32_t)nrows * C * 2);
        u32x4 raw[G::SLOTS];
#pragma unroll
        for (int s = 0; s < G::SLOTS; ++s) {
            const int r = wave * (G::TM / kPjWaves) + s * G::RPW + rs;
            raw[s] = bload16(rx, (uint32_t)(r * C + li * 8) * 2u);
        }
        // (empty resources without a LayerNorm: those loads read zeros and touch no memory)
        const rsrc_t rw = make_buf(a.lnw, a.lnw ? C * 4 : 0), rb = make_buf(a.lnb, a.lnb ? C * 4 : 0);
        float wv[8], bv[8];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const f32x4 w4 = __builtin_bit_cast(f32x4, bload16(rw, (uint32_t)(li * 8 + 4 * q) * 4u));
            const f32x4 b4 = __builtin_bit_cast(f32x4, bload16(rb, (uint32_t)(li * 8 + 4 * q) * 4u));
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                wv[4 * q + e] = w4[e];
                bv[4 * q + e] = b4[e];
            }
        }
        const bool stats = a.mean != nullptr && blockIdx.y == 0;  // one writer per token tile
        const rsrc_t rm = make_buf(stats ? a.mean + row0 : nullptr, stats ? (uint32_t)nrows * 4u : 0u);
        const rsrc_t rr = make_buf(stats ? a.rstd + row0 : nullptr, stats ? (uint32_t)nrows * 4u : 0u);
        constexpr float inv_c = 1.0f / (float)C;
        if (a.lnw == nullptr) {  // plain linear layer: the tile goes to LDS as it is
#pragma unroll
            for (int s = 0; s < G::SLOTS; ++s) {
                const int r = wave * (G::TM / kPjWaves) + s * G::RPW + rs;
                *(u32x4 *)(lds + r * G::STRIDE + li * 16) = raw[s];
            }
        } else {
#pragma unroll
        for (int s = 0; s < G::SLOTS; ++s) {
            const int r = wave * (G::TM / kPjWaves) + s * G::RPW + rs;
            float f[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                f[2 * i] = __uint_as_float(raw[s][i] << 16);
                f[2 * i + 1] = __uint_as_float(raw[s][i] & 0xffff0000u);
            }
            const float k0 = __shfl(f[0], lane & ~(G::LPR - 1), 64);
            float sum = 0.f;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                f[e] -= k0;
                sum += f[e];
            }
            const float mus = pj_row_sum<G::LPR>(sum) * inv_c;
            float ss = 0.f;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                f[e] -= mus;
                ss = fmaf(f[e], f[e], ss);
            }
            const float rstd = rsqrtf(pj_row_sum<G::LPR>(ss) * inv_c + a.eps);
            bf16x8 o;
#pragma unroll
            for (int e = 0; e < 8; ++e) o[e] = (__bf16)fmaf(f[e] * rstd, wv[e], bv[e]);
            *(bf16x8 *)(lds + r * G::STRIDE + li * 16) = o;
            const uint32_t so = li == 0 ? (uint32_t)r * 4u : kOOB;
            bstore4(__float_as_uint(k0 + mus), rm, so);
            bstore4(__float_as_uint(rstd), rr, so);
        }
        }
    }
    __syncthreads();

    // ---- the normalised tile itself, for the backward (optional) -----------
    if (a.y) {
        const rsrc_t ry = make_buf((char *)a.y + row0 * C * 2, (uint32_t)nrows * C * 2);
        constexpr int CH = C / 8;  // 16-byte chunks per row
        for (int idx = threadIdx.x; idx < G::TM * CH; idx += 64 * kPjWaves) {
            const int r = idx / CH, c = idx % CH;
            bstore16(*(const u32x4 *)(lds + r * G::STRIDE + c * 16), ry, (uint32_t)(r * C + c * 8) * 2u);
        }
    }

    // ---- 2./3. projections -------------------------------------------------
    const int n = lane & 31, h = lane >> 5;
    // feature tiles of this workgroup: group blockIdx.y of gridDim.y equal
    // contiguous groups (more than one only when the tokens alone would leave
    // CUs idle)
    const int NFall = a.P * a.HD / 32;
    const int per = (NFall + (int)gridDim.y - 1) / (int)gridDim.y;
    const int fbeg = (int)blockIdx.y * per;
    const int NF = NFall < fbeg + per ? NFall : fbeg + per;
    const rsrc_t rW = make_buf(a.W, (uint32_t)(a.P * a.HD) * C * 2u);
    const rsrc_t rB = make_buf(a.bias, a.bias ? (uint32_t)(a.P * a.HD) * 4u : 0u);
    int f = fbeg + wave;
    if (f >= NF) return;  // wave-uniform; no barrier follows

    for (; f < NF; f += kPjWaves) {
        // this tile's 32 weight rows as A fragments (all k-steps issued up
        // front and consumed in order; the other wave on the SIMD covers the
        // wait for the first)
        bf16x8 wcur[G::KS];
#pragma unroll
        for (int ks = 0; ks < G::KS; ++ks)
            wcur[ks] = __builtin_bit_cast(bf16x8, bload16(rW, (uint32_t)((f * 32 + n) * C + ks * 16 + 8 * h) * 2u));
        f32x4 bq[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) bq[j] = __builtin_bit_cast(f32x4, bload16(rB, (uint32_t)(f * 32 + 8 * j + 4 * h) * 4u));

        f32x16 acc[TB];
#pragma unroll
        for (int t = 0; t < TB; ++t)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[t][i] = 0.f;
        // token fragments one k-step ahead of the products; the scheduling
        // barrier keeps the compiler from hoisting every LDS read of the
        // tile (which would need TB*KS*4 registers)
        bf16x8 bcur[TB], bnxt[TB];
#pragma unroll
        for (int t = 0; t < TB; ++t) bcur[t] = *(const bf16x8 *)(lds + (t * 32 + n) * G::STRIDE + 16 * h);
#pragma unroll
        for (int ks = 0; ks < G::KS; ++ks) {
            if (ks + 1 < G::KS) {
#pragma unroll
                for (int t = 0; t < TB; ++t)
                    bnxt[t] = *(const bf16x8 *)(lds + (t * 32 + n) * G::STRIDE + (ks + 1) * 32 + 16 * h);
            }
#pragma unroll
            for (int t = 0; t < TB; ++t) acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wcur[ks], bcur[t], acc[t], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int t = 0; t < TB; ++t) bcur[t] = bnxt[t];
        }

        // epilogue through the wave's staging area: D[feature][token] goes in
        // as 8-byte pieces (4 features of a token), comes out as 16-byte
        // pieces of token rows, so each store covers 64 contiguous bytes of
        // 16 token rows
        const int p = (f * 32) / a.HD, fl = (f * 32) % a.HD;
        void *outp = p == 0 ? a.out0 : p == 1 ? a.out1 : p == 2 ? a.out2 : a.out3;
        const rsrc_t ro = make_buf((char *)outp + row0 * a.HD * 2, (uint32_t)nrows * a.HD * 2u);
        char *stage = lds + G::TM * G::STRIDE + wave * G::OBYTES;
#pragma unroll
        for (int t = 0; t < TB; ++t)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                __attribute__((ext_vector_type(4))) __bf16 o4;
#pragma unroll
                for (int e = 0; e < 4; ++e) o4[e] = (__bf16)(acc[t][4 * j + e] + bq[j][e]);
                *(u32x2 *)(stage + (t * 32 + n) * G::OSTRIDE + (8 * j + 4 * h) * 2) = __builtin_bit_cast(u32x2, o4);
            }
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int q = 0; q < G::TM / 16; ++q) {
            const int tok = q * 16 + (lane >> 2), ch = lane & 3;
            const u32x4 v = *(const u32x4 *)(stage + tok * G::OSTRIDE + ch * 16);
            bstore16(v, ro, (uint32_t)(tok * a.HD + fl + 8 * ch) * 2u);
        }
        __builtin_amdgcn_wave_barrier();
    }
}

template <int C, int TB>
hipError_t ln_proj_c(const PjArgs &a, hipStream_t s) {
    const int64_t tm = 32 * TB;
    const int64_t nwg = (a.R + tm - 1) / tm;
    // fewer token tiles than CUs: split the feature tiles over up to NF/8
    // workgroups per token tile (each recomputes the tile's LayerNorm)
    const int nf = a.P * a.HD / 32;
    int64_t fs = nwg < 256 ? 256 / nwg : 1;
    const int64_t fs_max = nf / kPjWaves > 1 ? nf / kPjWaves : 1;
    fs = fs < fs_max ? fs : fs_max;
    hipLaunchKernelGGL((ln_proj_kernel<C, TB>), dim3((unsigned)nwg, (unsigned)fs), dim3(64 * kPjWaves), 0, s, a);
    return hipGetLastError();
}

// tokens per workgroup: 128 (TB = 4) unless overridden (EVO_PROJ_TB = 2 or 4)
int proj_tb() {
    static const int tb = [] {
        const char *e = getenv("EVO_PROJ_TB");
        const int v = e ? atoi(e) : 0;
        return (v == 2 || v == 4) ? v : 4;
    }();
    return tb;
}

template <int C>
hipError_t ln_proj_tb(const PjArgs &a, hipStream_t s) {
    return proj_tb() == 2 ? ln_proj_c<C, 2>(a, s) : ln_proj_c<C, 4>(a, s);
}

}  // namespace

bool proj_supported(int C, int HD, int P) {
    return (C == 64 || C == 128 || C == 256) && HD >= 32 && HD <= 1024 && HD % 32 == 0 && P >= 1 && P <= 4;
}

hipError_t launch_ln_proj(const PjArgs &a, hipStream_t s) {
    switch (a.C) {
        case 64: return ln_proj_tb<64>(a, s);
        case 128: return ln_proj_tb<128>(a, s);
        case 256: return ln_proj_tb<256>(a, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace evo
