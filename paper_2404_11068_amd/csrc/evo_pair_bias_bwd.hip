// evo_pair_bias_bwd.hip -- backward of the pair-bias projection, gfx950.
//
// The forward (evo_pair_bias.hip) maps each layer-normalised pair entry
// y = LN(z[b, i, j, :]) to one logit bias per head, v[h] = sum_c y[c] W[h, c]
// (ScaleFold Section 3.3, the pair-bias term of the attention).  Given the
// attention backward's dL/dbias g[b, h, i, j] (fp32, in the forward's output
// layout), this computes
//
//   dY[c]   = sum_h g[h] W[h, c]                      per entry
//   dz      = LayerNorm backward of dY                 per entry, bf16
//   dW[h,c] = sum over entries of g[h] y[c]
//   dln_w   = sum over entries of dY * xhat,   dln_b = sum over entries of dY
//
// Persistent workgroups of 4 waves walk tiles of 4 rows i x TJ columns j
// (TJ = 64, 32, 16 for C = 64, 128, 256: eight entries per lane group).  The
// tile's g values (H x 4 x TJ floats) are staged in LDS from 16-byte loads in
// either layout; each wave then takes one row, an entry
// read by C/8 lanes (16 bytes each), recomputes the LayerNorm statistics as
// the forward does, and writes dz with 16-byte stores.  dW, dln_w and dln_b
// accumulate in registers over all of the workgroup's entries and are summed
// in a fixed order (lanes, then waves) into one partial row per workgroup; a
// second kernel adds the partial rows in workgroup order.  No atomics, so
// repeated calls give identical bits.
#include "evo_frag.h"
#include "evo_kernels.h"

namespace evo {
namespace {

constexpr int kPbbWaves = 4;   // rows i per tile, one per wave
constexpr int kPbbSL = 8;      // entries per lane group and tile (all loaded before the arithmetic)
constexpr int kPbbMaxWG = 512; // persistent grid (two workgroups per CU: the register budget allows two waves per SIMD)

// columns j per tile: eight wave slots of 64 / (C / 8) entries
__host__ __device__ constexpr int pbb_tj(int C) { return kPbbSL * (64 / (C / 8)); }

// sum over an LPR-lane group (DPP within 16-lane rows, a swizzle across them)
template <int LPR>
__device__ __forceinline__ float pbb_row_sum(float v) {
    if constexpr (LPR >= 2) v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
    if constexpr (LPR >= 4) v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, false));
    if constexpr (LPR >= 8) v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x141, 0xF, 0xF, false));
    if constexpr (LPR >= 16) v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x140, 0xF, 0xF, false));
    if constexpr (LPR >= 32) v += __shfl_xor(v, 16, 64);
    return v;
}

// sum over the lanes that hold the same channels (lane bits >= log2(LPR)),
// in a fixed butterfly order
template <int LPR>
__device__ __forceinline__ float pbb_group_sum(float v) {
#pragma unroll
    for (int m = LPR; m < 64; m *= 2) v += __shfl_xor(v, m, 64);
    return v;
}

template <int C, int H>
__global__ __launch_bounds__(64 * kPbbWaves) void pair_bias_bwd_kernel(PbBwdArgs a, int64_t n_tiles,
                                                                      float *__restrict__ part) {
    constexpr int LPR = C / 8;          // lanes per pair entry
    constexpr int PPS = 64 / LPR;       // entries per wave slot
    constexpr int SL = kPbbSL;          // slots per wave
    constexpr int TJ = pbb_tj(C);       // columns per tile
    constexpr int NX = H * C + 2 * C;   // partial row: dW, dln_w, dln_b
    __shared__ __attribute__((aligned(16))) float gst[H][kPbbWaves][TJ];
    __shared__ __attribute__((aligned(16))) float red[kPbbWaves][NX];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int li = lane % LPR, rs = lane / LPR;
    const int Li = a.Li, Lj = a.Lj;
    const int ntj = (Lj + TJ - 1) / TJ, nti = Li / kPbbWaves;
    constexpr float inv_c = 1.0f / (float)C;

    // this lane's 8 channels: LayerNorm weight and bias, every head's weight
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
    const rsrc_t rW = make_buf(a.W, H * C * 2);
    u32x4 wpk[H];  // bf16 pairs: channel 2k in the low half, 2k+1 in the high half
#pragma unroll
    for (int h = 0; h < H; ++h) wpk[h] = bload16(rW, (uint32_t)(h * C + li * 8) * 2u);

    float acc[H][8], dlw[8], dlb[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        dlw[e] = dlb[e] = 0.f;
#pragma unroll
        for (int h = 0; h < H; ++h) acc[h][e] = 0.f;
    }

    for (int64_t t = blockIdx.x; t < n_tiles; t += gridDim.x) {
        const int jt = (int)(t % ntj);
        const int64_t rest = t / ntj;
        const int it = (int)(rest % nti);
        const int64_t b = rest / nti;
        const int i0 = it * kPbbWaves, j0 = jt * TJ, i = i0 + wave;

        // g of this tile -> LDS (Li is a multiple of 8, so rows i0..i0+3 exist)
        const rsrc_t rg = make_buf(a.dbias + b * (int64_t)H * Li * Lj, (uint32_t)(H * Li * Lj) * 4u);
        if (!a.transpose) {
            // rows (h, i) of TJ columns: pieces of 4 columns
            constexpr int NPC = TJ / 4;
            for (int idx = tid; idx < H * kPbbWaves * NPC; idx += 64 * kPbbWaves) {
                const int h = idx / (kPbbWaves * NPC), w = (idx / NPC) % kPbbWaves, ch = idx % NPC;
                const int jj = j0 + 4 * ch;
                const u32x4 v = bload16(rg, jj < Lj ? (uint32_t)(((int64_t)h * Li + i0 + w) * Lj + jj) * 4u : kOOB);
                *(u32x4 *)&gst[h][w][4 * ch] = v;
            }
        } else {
            // rows (h, j): the tile's 4 rows i are 16 contiguous bytes
            for (int idx = tid; idx < H * TJ; idx += 64 * kPbbWaves) {
                const int h = idx / TJ, c = idx % TJ;
                const int jj = j0 + c;
                const f32x4 v = __builtin_bit_cast(
                    f32x4, bload16(rg, jj < Lj ? (uint32_t)(((int64_t)h * Lj + jj) * Li + i0) * 4u : kOOB));
#pragma unroll
                for (int w = 0; w < kPbbWaves; ++w) gst[h][w][c] = v[w];
            }
        }
        // this wave's row of z (entries past Lj read as zeros and are not written)
        const int64_t zrow = (b * Li + i) * (int64_t)Lj;
        const rsrc_t rz = make_buf((const char *)a.z + zrow * C * 2, (uint32_t)Lj * C * 2u);
        const rsrc_t rdz = make_buf((char *)a.dz + zrow * C * 2, (uint32_t)Lj * C * 2u);
        u32x4 raw[SL];
#pragma unroll
        for (int s = 0; s < SL; ++s) {
            const int j = j0 + s * PPS + rs;
            raw[s] = bload16(rz, j < Lj ? (uint32_t)(j * C + li * 8) * 2u : kOOB);
        }
        __syncthreads();

#pragma unroll
        for (int s = 0; s < SL; ++s) {
            float f[8];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                f[2 * q] = __uint_as_float(raw[s][q] << 16);
                f[2 * q + 1] = __uint_as_float(raw[s][q] & 0xffff0000u);
            }
            // statistics as in the forward: shift by the entry's first value,
            // mean, then the variance of the centred values
            const float k0 = __shfl(f[0], lane & ~(LPR - 1), 64);
            float sum = 0.f;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                f[e] -= k0;
                sum += f[e];
            }
            const float mus = pbb_row_sum<LPR>(sum) * inv_c;
            float ss = 0.f;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                f[e] -= mus;
                ss = fmaf(f[e], f[e], ss);
            }
            const float rstd = rsqrtf(pbb_row_sum<LPR>(ss) * inv_c + a.eps);
            const int p = s * PPS + rs;
            float g[H];
#pragma unroll
            for (int h = 0; h < H; ++h) g[h] = gst[h][wave][p];
            float xh[8], dy[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                xh[e] = f[e] * rstd;
                dy[e] = 0.f;
            }
#pragma unroll
            for (int h = 0; h < H; ++h) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float w0 = __uint_as_float(wpk[h][q] << 16), w1 = __uint_as_float(wpk[h][q] & 0xffff0000u);
                    dy[2 * q] = fmaf(g[h], w0, dy[2 * q]);
                    dy[2 * q + 1] = fmaf(g[h], w1, dy[2 * q + 1]);
                }
            }
            float s1 = 0.f, s2 = 0.f;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float y = fmaf(xh[e], wv[e], bv[e]);
#pragma unroll
                for (int h = 0; h < H; ++h) acc[h][e] = fmaf(g[h], y, acc[h][e]);
                dlw[e] = fmaf(dy[e], xh[e], dlw[e]);
                dlb[e] += dy[e];
                const float wd = wv[e] * dy[e];
                s1 += wd;
                s2 = fmaf(wd, xh[e], s2);
            }
            const float m1 = pbb_row_sum<LPR>(s1) * inv_c, m2 = pbb_row_sum<LPR>(s2) * inv_c;
            u32x4 out;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float d0 = rstd * (wv[2 * q] * dy[2 * q] - fmaf(xh[2 * q], m2, m1));
                const float d1 = rstd * (wv[2 * q + 1] * dy[2 * q + 1] - fmaf(xh[2 * q + 1], m2, m1));
                out[q] = (uint32_t)f2bf(d0) | ((uint32_t)f2bf(d1) << 16);
            }
            const int j = j0 + p;
            bstore16(out, rdz, j < Lj ? (uint32_t)(j * C + li * 8) * 2u : kOOB);
        }
        __syncthreads();  // the next tile overwrites gst
    }

    // partial row of this workgroup: lanes holding the same channels, then
    // the four waves, each in a fixed order
#pragma unroll
    for (int e = 0; e < 8; ++e) {
#pragma unroll
        for (int h = 0; h < H; ++h) acc[h][e] = pbb_group_sum<LPR>(acc[h][e]);
        dlw[e] = pbb_group_sum<LPR>(dlw[e]);
        dlb[e] = pbb_group_sum<LPR>(dlb[e]);
    }
    if (rs == 0) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
#pragma unroll
            for (int h = 0; h < H; ++h) {
                const f32x4 v = {acc[h][4 * q], acc[h][4 * q + 1], acc[h][4 * q + 2], acc[h][4 * q + 3]};
                *(f32x4 *)&red[wave][h * C + li * 8 + 4 * q] = v;
            }
            const f32x4 vw = {dlw[4 * q], dlw[4 * q + 1], dlw[4 * q + 2], dlw[4 * q + 3]};
            const f32x4 vb = {dlb[4 * q], dlb[4 * q + 1], dlb[4 * q + 2], dlb[4 * q + 3]};
            *(f32x4 *)&red[wave][H * C + li * 8 + 4 * q] = vw;
            *(f32x4 *)&red[wave][H * C + C + li * 8 + 4 * q] = vb;
        }
    }
    __syncthreads();
    const rsrc_t rp = make_buf(part + (int64_t)blockIdx.x * NX, NX * 4);
    for (int x = tid; x < NX; x += 64 * kPbbWaves) {
        float v = red[0][x];
#pragma unroll
        for (int w = 1; w < kPbbWaves; ++w) v += red[w][x];
        bstore4(__float_as_uint(v), rp, (uint32_t)x * 4u);
    }
}

// out = sum over workgroups of the partial rows, in a fixed order: a block
// takes 4 groups of four columns and splits the rows into 64 interleaved
// slices, whose sums are then added in slice order (80 blocks at C = 128,
// H = 8: 16 groups per block left the partial rows to 20 CUs, 4.8 us against
// 4.0 us)
__global__ __launch_bounds__(256) void pb_param_reduce_kernel(const float *__restrict__ part, int n_part, int HC,
                                                             int C, float *__restrict__ dW, float *__restrict__ dlw,
                                                             float *__restrict__ dlb) {
    constexpr int KS = 64, QB = 4;
    __shared__ f32x4 sred[KS][QB];
    const int ks = threadIdx.x / QB, qb = threadIdx.x % QB;
    const int NX = HC + 2 * C;
    const int x4 = (blockIdx.x * QB + qb) * 4;
    const bool ok = x4 < NX;
    const rsrc_t rp = make_buf(part, (uint32_t)n_part * NX * 4u);
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
    int k = ks;
    for (; k + 3 * KS < n_part; k += 4 * KS) {  // four loads in flight, added in k order
        f32x4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            v[u] = __builtin_bit_cast(f32x4, bload16(rp, ok ? (uint32_t)((k + u * KS) * NX + x4) * 4u : kOOB));
#pragma unroll
        for (int u = 0; u < 4; ++u) s += v[u];
    }
    for (; k < n_part; k += KS) s += __builtin_bit_cast(f32x4, bload16(rp, ok ? (uint32_t)(k * NX + x4) * 4u : kOOB));
    sred[ks][qb] = s;
    __syncthreads();
    if (ks != 0 || !ok) return;
    s = sred[0][qb];
#pragma unroll
    for (int j = 1; j < KS; ++j) s += sred[j][qb];
    float *dst = x4 < HC ? dW + x4 : x4 < HC + C ? dlw + (x4 - HC) : dlb + (x4 - HC - C);
    *(f32x4 *)dst = s;
}

template <int C, int H>
hipError_t launch_ch(const PbBwdArgs &a, void *ws, hipStream_t s) {
    const int64_t n_tiles = a.B * (a.Li / kPbbWaves) * ((a.Lj + pbb_tj(C) - 1) / pbb_tj(C));
    const int64_t nwg = pair_bias_bwd_workgroups(a.B, a.Li, a.Lj, C);
    float *part = (float *)ws;
    hipLaunchKernelGGL((pair_bias_bwd_kernel<C, H>), dim3((unsigned)nwg), dim3(64 * kPbbWaves), 0, s, a, n_tiles,
                       part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int nx4 = (H * C + 2 * C) / 4;
    hipLaunchKernelGGL(pb_param_reduce_kernel, dim3((unsigned)((nx4 + 3) / 4)), dim3(256), 0, s, part, (int)nwg,
                       H * C, C, a.dW, a.dlnw, a.dlnb);
    return hipGetLastError();
}

template <int C>
hipError_t launch_c(const PbBwdArgs &a, void *ws, hipStream_t s) {
    switch (a.H) {
        case 1: return launch_ch<C, 1>(a, ws, s);
        case 2: return launch_ch<C, 2>(a, ws, s);
        case 4: return launch_ch<C, 4>(a, ws, s);
        case 8: return launch_ch<C, 8>(a, ws, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace

bool pair_bias_bwd_supported(int C, int H) {
    return (C == 64 || C == 128 || C == 256) && (H == 1 || H == 2 || H == 4 || H == 8);
}

int64_t pair_bias_bwd_workgroups(int64_t B, int Li, int Lj, int C) {
    const int tj = pbb_tj(C);
    const int64_t n_tiles = B * (Li / kPbbWaves) * ((Lj + tj - 1) / tj);
    return n_tiles < kPbbMaxWG ? (n_tiles > 0 ? n_tiles : 1) : kPbbMaxWG;
}

size_t pair_bias_bwd_workspace(int64_t B, int Li, int Lj, int C, int H) {
    return (size_t)pair_bias_bwd_workgroups(B, Li, Lj, C) * (size_t)(H * C + 2 * C) * 4;
}

hipError_t launch_pair_bias_bwd(const PbBwdArgs &a, void *ws, hipStream_t s) {
    switch (a.C) {
        case 64: return launch_c<64>(a, ws, s);
        case 128: return launch_c<128>(a, ws, s);
        case 256: return launch_c<256>(a, ws, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace evo
