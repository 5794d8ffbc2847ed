// evo_pair_bias.hip -- LayerNorm of the pair representation projected to one
// logit bias per head, written in the attention's bias layout, gfx950.
//
// The pair bias that ScaleFold Section 3.3 adds to the attention logits is a
// bias-free linear map of the layer-normalised pair entry z[b, i, j, :] to H
// values.  This kernel computes it and writes bias[b, h, i, j] (or, for
// triangle attention around the ending node, bias[b, h, j, i]) directly, so
// the [B, Li, Lj, H] intermediate and its transpose never reach HBM.
//
// Workgroup = 4 waves = 4 rows i of one batch entry times 16 columns j.  In a
// wave, a pair entry of C channels is read by LPR = C / 8 lanes (16 bytes
// each; all the wave's loads are issued before any arithmetic).  LayerNorm
// statistics come from DPP row reductions; the normalised entry is rounded
// to bf16 and each head's dot product is four v_dot2_f32_bf16 per lane; the
// H partial sums are then reduce-scattered over the entry's lanes (each lane
// ends with the full sum of one head, or of H/LPR heads).  The H x 4 x 16
// results go through LDS so that the stores cover 16 contiguous bytes (plain
// layout) or 8 (transposed).  Lengths are multiples of 8, so no 16- or 8-byte
// piece straddles a row.  Sixteen columns per workgroup (not 32) give four
// waves per SIMD at the 256 x 256 crop, which hides more of each wave's
// single batch of loads (pair_bias_kernel<128, 8>: 9.3 -> 8.4 us mean).
#include "evo_frag.h"
#include "evo_kernels.h"

namespace evo {
namespace {

constexpr int kPbWaves = 4;  // rows i per workgroup, one per wave
constexpr int kPbTJ = 16;    // columns j per workgroup

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;

template <int LPR>
__device__ __forceinline__ float pb_row_sum(float v) {
    if constexpr (LPR >= 2) v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
    if constexpr (LPR >= 4) v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, false));
    if constexpr (LPR >= 8) v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x141, 0xF, 0xF, false));
    if constexpr (LPR >= 16) v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x140, 0xF, 0xF, false));
    if constexpr (LPR >= 32) v += __shfl_xor(v, 16, 64);
    return v;
}

// value of the partner lane at distance M inside an LPR-lane group: xor 16
// crosses 16-lane rows (ds_bpermute); 8 and 4 use the row and half-row
// mirrors (partner 15-i, 7-i: the bit M differs and every higher bit is
// shared, which is all the reductions below need); 2 and 1 swap pairs.
template <int M>
__device__ __forceinline__ float pb_partner(float v) {
    if constexpr (M == 16) return __shfl_xor(v, 16, 64);
    constexpr int ctrl = M == 8 ? 0x140 : M == 4 ? 0x141 : M == 2 ? 0x4E : 0xB1;
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), ctrl, 0xF, 0xF, false));
}

// Reduce-scatter of H per-lane partial sums over an LPR-lane group: at each
// lane bit (highest first) the lanes split their current set of heads in
// halves, keep one half and add the partner's values for it (sending the
// other half); once one head is left the remaining bits are plain pairwise
// sums.  Afterwards the lane holds the full sums of heads [*first, *first +
// KEEP) with KEEP = max(1, H / LPR).  Cost: about H + log2(LPR) exchanges
// instead of H * log2(LPR) for one full reduction per head.
template <int LPR, int H, int M = LPR / 2, int CNT = H>
__device__ __forceinline__ void pb_reduce_scatter(float (&v)[H], int li, int *first) {
    if constexpr (M >= 1) {
        if constexpr (CNT > 1) {
            constexpr int HALF = CNT / 2;
            const bool upper = (li & M) != 0;
#pragma unroll
            for (int k = 0; k < HALF; ++k) {
                const float send = upper ? v[k] : v[HALF + k];
                const float keep = upper ? v[HALF + k] : v[k];
                v[k] = keep + pb_partner<M>(send);
            }
            if (upper) *first += HALF;
            pb_reduce_scatter<LPR, H, M / 2, HALF>(v, li, first);
        } else {
            v[0] += pb_partner<M>(v[0]);
            pb_reduce_scatter<LPR, H, M / 2, 1>(v, li, first);
        }
    }
}

__device__ __forceinline__ void bstore8(u32x2 v, rsrc_t r, uint32_t off) {
    __builtin_amdgcn_raw_buffer_store_b64(v, r, off, 0, 0);
}

template <int C, int H>
__global__ __launch_bounds__(64 * kPbWaves) void pair_bias_kernel(PbArgs a) {
    constexpr int LPR = C / 8;          // lanes per pair entry
    constexpr int PPS = 64 / LPR;       // entries per wave slot
    constexpr int SL = kPbTJ / PPS;     // slots per wave
    __shared__ __attribute__((aligned(16))) uint16_t stage[H][kPbWaves][kPbTJ];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int li = lane % LPR, rs = lane / LPR;
    const int64_t b = blockIdx.z;
    const int i0 = blockIdx.y * kPbWaves, i = i0 + wave;
    const int j0 = blockIdx.x * kPbTJ;
    const int Li = a.Li, Lj = a.Lj;

    // row (b, i) of z: Lj entries of C channels; a row past Li is empty
    const bool row_ok = i < Li;
    const int64_t zrow = (b * Li + i) * (int64_t)Lj;
    const rsrc_t rz = make_buf(row_ok ? (const char *)a.z + zrow * C * 2 : nullptr,
                               row_ok ? (uint32_t)Lj * C * 2u : 0u);
    u32x4 raw[SL];
#pragma unroll
    for (int s = 0; s < SL; ++s) {
        const int j = j0 + s * PPS + rs;
        raw[s] = bload16(rz, j < Lj ? (uint32_t)(j * C + li * 8) * 2u : kOOB);
    }
    const rsrc_t rw = make_buf(a.lnw, C * 4), rb = make_buf(a.lnb, C * 4);
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
    // this lane's 8 channels of every head's weight row, as bf16 pairs
    const rsrc_t rW = make_buf(a.W, H * C * 2);
    bf16x2 wh[H][4];
#pragma unroll
    for (int h = 0; h < H; ++h) {
        // bit-cast the whole vector, then take components (a bit-cast of a
        // single vector component reads component 0 with this compiler)
        const bf16x8 v = __builtin_bit_cast(bf16x8, bload16(rW, (uint32_t)(h * C + li * 8) * 2u));
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            wh[h][q][0] = v[2 * q];
            wh[h][q][1] = v[2 * q + 1];
        }
    }
    const bool stats = a.mean != nullptr;
    const rsrc_t rm = make_buf(stats && row_ok ? a.mean + zrow : nullptr, stats && row_ok ? (uint32_t)Lj * 4u : 0u);
    const rsrc_t rr = make_buf(stats && row_ok ? a.rstd + zrow : nullptr, stats && row_ok ? (uint32_t)Lj * 4u : 0u);
    constexpr float inv_c = 1.0f / (float)C;

#pragma unroll
    for (int s = 0; s < SL; ++s) {
        float f[8];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            f[2 * q] = __uint_as_float(raw[s][q] << 16);
            f[2 * q + 1] = __uint_as_float(raw[s][q] & 0xffff0000u);
        }
        const float k0 = __shfl(f[0], lane & ~(LPR - 1), 64);
        float sum = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            f[e] -= k0;
            sum += f[e];
        }
        const float mus = pb_row_sum<LPR>(sum) * inv_c;
        float ss = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            f[e] -= mus;
            ss = fmaf(f[e], f[e], ss);
        }
        const float rstd = rsqrtf(pb_row_sum<LPR>(ss) * inv_c + a.eps);
        bf16x2 y[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            y[q][0] = (__bf16)fmaf(f[2 * q] * rstd, wv[2 * q], bv[2 * q]);
            y[q][1] = (__bf16)fmaf(f[2 * q + 1] * rstd, wv[2 * q + 1], bv[2 * q + 1]);
        }
        // one partial dot product per head over this lane's 8 channels, then
        // a reduce-scatter over the entry's lanes
        float dh[H];
#pragma unroll
        for (int h = 0; h < H; ++h) {
            float d = 0.f;
#pragma unroll
            for (int q = 0; q < 4; ++q) d = __builtin_amdgcn_fdot2_f32_bf16(y[q], wh[h][q], d, false);
            dh[h] = d;
        }
        int first = 0;
        pb_reduce_scatter<LPR, H>(dh, li, &first);
        constexpr int KEEP = H > LPR ? H / LPR : 1;
        // lanes that differ only in the bits summed after the split hold the
        // same heads: the one with those bits clear writes them
        constexpr int DUP = H >= LPR ? 1 : LPR / H;
        const int p = s * PPS + rs;
        if ((li & (DUP - 1)) == 0) {
#pragma unroll
            for (int k = 0; k < KEEP; ++k) stage[first + k][wave][p] = __builtin_bit_cast(uint16_t, (__bf16)dh[k]);
        }
        const int j = j0 + p;
        const uint32_t so = (li == 0 && j < Lj) ? (uint32_t)j * 4u : kOOB;
        bstore4(__float_as_uint(k0 + mus), rm, so);
        bstore4(__float_as_uint(rstd), rr, so);
    }
    __syncthreads();

    const rsrc_t ro = make_buf((char *)a.out + b * H * (int64_t)Li * Lj * 2, (uint32_t)(H * Li * Lj) * 2u);
    if (!a.transpose) {
        // rows (h, i) of kPbTJ columns: pieces of 8 columns
        constexpr int NPC = kPbTJ / 8;
        for (int idx = threadIdx.x; idx < H * kPbWaves * NPC; idx += 64 * kPbWaves) {
            const int h = idx / (kPbWaves * NPC), w = (idx / NPC) % kPbWaves, ch = idx % NPC;
            const u32x4 v = *(const u32x4 *)&stage[h][w][ch * 8];
            const int ii = i0 + w, jj = j0 + ch * 8;
            const bool ok = ii < Li && jj < Lj;
            bstore16(v, ro, ok ? (uint32_t)(((int64_t)h * Li + ii) * Lj + jj) * 2u : kOOB);
        }
    } else {
        // rows (h, j) of the 4 rows i of this workgroup: 8 bytes each
        for (int idx = threadIdx.x; idx < H * kPbTJ; idx += 64 * kPbWaves) {
            const int h = idx / kPbTJ, c = idx % kPbTJ;
            u32x2 v;
            v[0] = (uint32_t)stage[h][0][c] | ((uint32_t)stage[h][1][c] << 16);
            v[1] = (uint32_t)stage[h][2][c] | ((uint32_t)stage[h][3][c] << 16);
            const int jj = j0 + c;
            const bool ok = i0 < Li && jj < Lj;
            bstore8(v, ro, ok ? (uint32_t)(((int64_t)h * Lj + jj) * Li + i0) * 2u : kOOB);
        }
    }
}

template <int C, int H>
hipError_t pair_bias_ch(const PbArgs &a, hipStream_t s) {
    const dim3 grid((unsigned)((a.Lj + kPbTJ - 1) / kPbTJ), (unsigned)((a.Li + kPbWaves - 1) / kPbWaves),
                    (unsigned)a.B);
    hipLaunchKernelGGL((pair_bias_kernel<C, H>), grid, dim3(64 * kPbWaves), 0, s, a);
    return hipGetLastError();
}

template <int C>
hipError_t pair_bias_c(const PbArgs &a, hipStream_t s) {
    switch (a.H) {
        case 1: return pair_bias_ch<C, 1>(a, s);
        case 2: return pair_bias_ch<C, 2>(a, s);
        case 4: return pair_bias_ch<C, 4>(a, s);
        case 8: return pair_bias_ch<C, 8>(a, s);
        case 16: return pair_bias_ch<C, 16>(a, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace

bool pair_bias_supported(int C, int H) {
    return (C == 64 || C == 128 || C == 256) && (H == 1 || H == 2 || H == 4 || H == 8 || H == 16);
}

hipError_t launch_pair_bias(const PbArgs &a, hipStream_t s) {
    switch (a.C) {
        case 64: return pair_bias_c<64>(a, s);
        case 128: return pair_bias_c<128>(a, s);
        case 256: return pair_bias_c<256>(a, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace evo
