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

// Row padding (bf16 elements) of the LDS tiles read with the transposing LDS
// read.  Per 32 lanes that read takes 64 contiguous bytes from each of four
// consecutive rows; it is conflict-free when the four rows fall in distinct
// 64-byte groups of the 64 four-byte banks.  With 32 elements of padding the
// row stride is 16 or 48 dwords past a multiple of 64 for every width used
// here but 32 (which keeps a two-way conflict).  Padding by 8 left two-way
// conflicts on every read: 6.4M conflict cycles per call at 32768 tokens x
// 256 channels, against 0.13M now.
constexpr int kLdsPad = 32;

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// workgroups of the weight-gradient pass (about one per CU)
inline int proj_bwd_dw_wgs() {
    static const int v = [] {
        const char *e = getenv("EVO_PROJ_DW_WGS");
        const int x = e ? atoi(e) : 0;
        return x >= 8 && x <= 65536 ? x : 256;
    }();
    return v;
}

// features per workgroup of the weight-gradient pass: 64, or 128 when C = 64
// (at least eight 32x32 output tiles, one per wave).  A block lies inside one
// projection (FB divides HD) or covers whole projections (HD divides FB, FB
// divides P*HD); 32 always qualifies (HD is a multiple of 32).
inline int proj_bwd_fb(int C, int HD, int P) {
    const int want = C == 64 ? 128 : 64;
    for (int fb = want; fb > 32; fb /= 2)
        if (HD % fb == 0 || (fb % HD == 0 && (P * HD) % fb == 0)) return fb;
    return 32;
}

// a wave-uniform pointer, moved to scalar registers
__device__ __forceinline__ const char *uniform_ptr(const char *p) {
    const uint64_t v = (uint64_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v), hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return (const char *)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ const void *dout_ptr(const PjBwdArgs &a, int p) {
    return p == 0 ? a.dout0 : p == 1 ? a.dout1 : p == 2 ? a.dout2 : a.dout3;
}

// ---------------------------------------------------------------------------
// dY tile of 128 tokens x C channels with NW = 16 waves (8 for C = 64).
// Output tiles (token tile tb, channel tile ct): wave w takes tb = w % 4 and
// ct = w / 4 + (NW / 4) j.  The contraction runs over stages of 64 features;
// both operands of a stage go through LDS (double-buffered): the dout rows
// [128 tokens][64 features], read back as row fragments, and the weight rows
// [64 features][C], read back with the transposing read.  Global loads of a
// stage are issued four stages ahead into a ring of register stages, in one
// in-order stream (the memory counter retires loads in issue order, so a
// wait for one load is a wait for every older one).
// A workgroup covers CW of the C channels (CW < C splits the channels over
// blockIdx.y when there are too few token blocks to fill the GPU).
template <int CW>
struct DyCfg {
    static constexpr int NW = CW >= 128 ? 16 : 8;
    static constexpr int NT = 64 * NW;
};

template <int C, int CW>
__global__ __launch_bounds__(DyCfg<CW>::NT) void dy_kernel(PjBwdArgs a, void *__restrict__ dy) {
    constexpr int NW = DyCfg<CW>::NW, NT = DyCfg<CW>::NT;
    constexpr int TM = 128, KC = 64, NR = 4;
    constexpr int NCT = CW / 32, CG = NW / 4, TPW = NCT / CG;  // channel tiles per wave
    static_assert(TPW >= 1 && NCT % CG == 0 && C % CW == 0, "dy_kernel takes C = 64, 128, 256");
    constexpr int WSTR = CW + kLdsPad;        // weight stage row stride (elements)
    // dout stage row stride: 36 dwords, so 16 lanes on 16 consecutive rows and
    // one 16-byte column hit 16 distinct groups of four banks
    constexpr int ASTR = KC + 8;
    constexpr int NA = TM * KC / 8 / NT;      // dout 16-byte chunks per thread and stage
    constexpr int NWL = KC * CW / 8 / NT;     // weight 16-byte chunks per thread and stage
    constexpr int OSTR = 40;                  // staging row stride (elements) of a 32x32 output tile
    constexpr int LW = KC * WSTR, LA = TM * ASTR;
    constexpr int LT = 2 * (LW + LA), LS = NW * 32 * OSTR;
    static_assert(NA >= 1 && NWL >= 1 && NA * NT == TM * KC / 8 && NWL * NT == KC * CW / 8, "stage split");
    __shared__ __attribute__((aligned(16))) uint16_t lds[LT > LS ? LT : LS];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 31, h = lane >> 5;
    const int tb = wave & 3, cg = wave >> 2;
    const int64_t row0 = (int64_t)blockIdx.x * TM;
    int64_t nrows = a.R - row0;
    nrows = nrows < TM ? nrows : TM;
    const int F = a.P * a.HD;
    const int NS = (F + KC - 1) / KC;
    const rsrc_t rW = make_buf(a.W, (uint32_t)F * C * 2u);
    const int c0 = blockIdx.y * CW;          // first channel of this workgroup

    // dout chunk j of this thread: k32 step (half) hf of the stage, token row
    // r, 16-byte column c4; a wave covers 16 rows x 4 columns of one half
    // (one projection), 16 lanes per column
    int a_r[NA], a_c4[NA], a_hf[NA];
#pragma unroll
    for (int j = 0; j < NA; ++j) {
        const int idx = tid + j * NT;
        a_hf[j] = idx >> 9;
        const int ii = idx & 511;
        a_r[j] = (ii >> 6) * 16 + (ii & 15);
        a_c4[j] = (ii >> 4) & 3;
    }
    // per-half cursor over the projections (wave-uniform, in scalar registers:
    // a per-lane copy would turn every load into a loop over distinct
    // resources): projection pointer, its successors, feature offset
    const uint32_t ablk = (uint32_t)nrows * a.HD * 2u;
    const int64_t aoff = row0 * a.HD * 2;
    const char *dp0 = (const char *)a.dout0 + aoff, *dp1 = (const char *)a.dout1 + aoff;
    const char *dp2 = (const char *)a.dout2 + aoff, *dp3 = (const char *)a.dout3 + aoff;
    const char *cur[NA], *nx1[NA], *nx2[NA], *nx3[NA];
    int lp[NA], lfl[NA];
#pragma unroll
    for (int j = 0; j < NA; ++j) {
        // k32 step a_hf[j] of stage 0: feature 32 a_hf[j]
        const int f = 32 * a_hf[j];
        const int p0 = __builtin_amdgcn_readfirstlane(f / a.HD);
        lfl[j] = __builtin_amdgcn_readfirstlane(f % a.HD);
        lp[j] = p0;
        cur[j] = uniform_ptr(p0 == 0 ? dp0 : p0 == 1 ? dp1 : p0 == 2 ? dp2 : dp3);
        nx1[j] = uniform_ptr(p0 == 0 ? dp1 : p0 == 1 ? dp2 : dp3);
        nx2[j] = uniform_ptr(p0 == 0 ? dp2 : dp3);
        nx3[j] = dp3;
    }
    auto advance = [&](int j) {  // by one stage (64 features = two k32 steps)
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            lfl[j] += 32;
            const bool wrap = lfl[j] == a.HD;
            lfl[j] = __builtin_amdgcn_readfirstlane(wrap ? 0 : lfl[j]);
            lp[j] = __builtin_amdgcn_readfirstlane(wrap ? lp[j] + 1 : lp[j]);
            cur[j] = uniform_ptr(wrap ? nx1[j] : cur[j]);
            nx1[j] = uniform_ptr(wrap ? nx2[j] : nx1[j]);
            nx2[j] = uniform_ptr(wrap ? nx3[j] : nx2[j]);
        }
    };
    auto load_stage = [&](int s, u32x4 (&ra)[NA], u32x4 (&rw)[NWL]) {
#pragma unroll
        for (int j = 0; j < NA; ++j) {
            const rsrc_t ro = make_buf(cur[j], __builtin_amdgcn_readfirstlane(lp[j] < a.P ? ablk : 0u));
            ra[j] = bload16(ro, (uint32_t)(a_r[j] * a.HD + lfl[j] + 8 * a_c4[j]) * 2u);
            advance(j);
        }
#pragma unroll
        for (int j = 0; j < NWL; ++j) {  // weight rows s*KC .. (rows past F read as zeros)
            const int idx = tid + j * NT;
            const int rr = idx / (CW / 8), c8 = idx % (CW / 8);
            rw[j] = bload16(rW, (uint32_t)((s * KC + rr) * C + c0 + c8 * 8) * 2u);
        }
    };
    auto store_stage = [&](int buf, const u32x4 (&ra)[NA], const u32x4 (&rw)[NWL]) {
        uint16_t *al = lds + buf * (LW + LA) + LW;
        uint16_t *wl = lds + buf * (LW + LA);
#pragma unroll
        for (int j = 0; j < NA; ++j)
            *(u32x4 *)&al[a_r[j] * ASTR + 32 * a_hf[j] + 8 * a_c4[j]] = ra[j];
#pragma unroll
        for (int j = 0; j < NWL; ++j) {
            const int idx = tid + j * NT;
            const int rr = idx / (CW / 8), c8 = idx % (CW / 8);
            *(u32x4 *)&wl[rr * WSTR + c8 * 8] = rw[j];
        }
    };

    f32x16 acc[TPW];
#pragma unroll
    for (int j = 0; j < TPW; ++j) acc[j] = zero16();
    u32x4 ra[NR][NA], rw[NR][NWL];
#pragma unroll
    for (int u = 0; u < NR; ++u) load_stage(u, ra[u], rw[u]);
    store_stage(0, ra[0], rw[0]);
    load_stage(NR, ra[0], rw[0]);
    __syncthreads();
    for (int s0 = 0; s0 < NS; s0 += NR) {
#pragma unroll
        for (int u = 0; u < NR; ++u) {
            const int s = s0 + u;
            const uint16_t *wl = lds + (u & 1) * (LW + LA);
            const uint16_t *al = wl + LW;
            if (s < NS) {
#pragma unroll
                for (int t = 0; t < 2; ++t) {
                    const Tr<bf16_t>::K32 af = load_k32<bf16_t>(&al[(tb * 32 + n) * ASTR + 32 * t], h);
#pragma unroll
                    for (int j = 0; j < TPW; ++j) {
                        const Tr<bf16_t>::K32 bf = load_k32_tr(&wl[(cg + CG * j) * 32], WSTR, 32 * t, 32, lane);
                        Tr<bf16_t>::mma_k32(acc[j], af, bf);
                    }
                }
            }
            // stage s+1 (loaded NR stages ago) into the other buffer; its
            // register stage then takes stage s+1+NR
            const int un = (u + 1) % NR;
            store_stage((u + 1) & 1, ra[un], rw[un]);
            load_stage(s + 1 + NR, ra[un], rw[un]);
            __syncthreads();
        }
    }

    // epilogue: D[token rho(i,h)][channel ct*32 + sig(n)] -> bf16 -> token rows
    const rsrc_t rd = make_buf((char *)dy + row0 * C * 2, (uint32_t)nrows * C * 2);
    uint16_t *st = lds + wave * 32 * OSTR;
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
        const int ct = cg + CG * j;
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
            bstore16(v, rd, (uint32_t)((tb * 32 + t) * C + c0 + ct * 32 + c4 * 8) * 2u);
        }
        __builtin_amdgcn_wave_barrier();
    }
}

// ---------------------------------------------------------------------------
// Partial dW (FB features x C channels) and dbias over one chunk of tokens.
// Tokens go through LDS 32 at a time (dout [32][FB] and y [32][C] rows,
// double-buffered); their global loads run through a ring of four register
// stages, issued four sub-blocks before the sub-block is staged.  The block
// has 16 waves when its (FB/32) x (C/32) tile grid has 16 tiles or more, else
// 8; wave w owns TPW consecutive tiles, all in one feature tile, so its dout
// fragment serves all of them.  One wave per feature tile (spread over the
// SIMDs) also sums dbias through an all-ones operand.  A feature block may
// span projections (FB > HD): its dout columns are loaded per projection
// segment, each segment by whole waves.  With `xcd_map`, the feature blocks
// of one token chunk are placed on one XCD (workgroups are dealt to the eight
// XCDs in turn), so that chunk's y rows are fetched into that XCD's L2 once.
template <int C, int FB>
struct DwCfg {
    static constexpr int NTILE = (FB / 32) * (C / 32);
    static constexpr int NW = NTILE >= 16 ? 16 : 8;
    static constexpr int NT = 64 * NW;
};

template <int C, int FB>
__global__ __launch_bounds__((DwCfg<C, FB>::NT)) void dw_kernel(PjBwdArgs a, int64_t chunk_tokens, int nfb,
                                                            int xcd_map, float *__restrict__ part_w,
                                                            float *__restrict__ part_b) {
    constexpr int NW = DwCfg<C, FB>::NW, NT = DwCfg<C, FB>::NT;
    constexpr int NFT = FB / 32, NCT = C / 32, NTILE = NFT * NCT;
    constexpr int TPW = NTILE / NW > 0 ? NTILE / NW : 1;
    constexpr int WPF = NCT / TPW;            // waves per feature tile
    constexpr int NR = 4;
    constexpr int DSTR = FB + kLdsPad, YSTR = C + kLdsPad;
    constexpr int ND = (32 * FB / 8 + NT - 1) / NT;
    constexpr int NY = (32 * C / 8 + NT - 1) / NT;
    __shared__ __attribute__((aligned(16))) uint16_t dl[2][32 * DSTR];
    __shared__ __attribute__((aligned(16))) uint16_t yl[2][32 * YSTR];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 31, h = lane >> 5;
    const int F = a.P * a.HD;
    const int L = blockIdx.x;
    int fb, chunk_i;
    if (xcd_map) {
        const int j = L >> 3;
        fb = j % nfb;
        chunk_i = (L & 7) + 8 * (j / nfb);
    } else {
        fb = L % nfb;
        chunk_i = L / nfb;
    }
    const int64_t chunk = chunk_i;
    const int64_t t_begin = chunk * chunk_tokens;
    int64_t t_end = t_begin + chunk_tokens;
    t_end = t_end < a.R ? t_end : a.R;
    const int f0 = fb * FB;
    const int ft = wave / WPF, ct0 = (wave % WPF) * TPW;
    const bool active = ft < NFT;
    const bool bias_owner = active && (wave % WPF) == ft % WPF;

    // dout chunk j of this thread: segment (projection) seg of the block,
    // token row r, 16-byte column c; segments are `segw` features wide and
    // 4 segw chunks long, a multiple of 64, so each wave loads one projection
    const int segw = FB <= a.HD ? FB : a.HD;
    const char *d_base[ND];
    int d_off[ND], d_lds[ND];
#pragma unroll
    for (int j = 0; j < ND; ++j) {
        const int idx = tid + j * NT;
        const int per = 4 * segw;           // chunks per segment: 32 rows x segw / 8
        const int seg = idx / per, rem = idx % per;
        const int r = rem / (segw / 8), c = rem % (segw / 8);
        const int f = f0 + seg * segw;      // first feature of the segment
        const int pj = __builtin_amdgcn_readfirstlane(f / a.HD);
        d_base[j] = uniform_ptr((const char *)dout_ptr(a, pj < a.P ? pj : 0));
        const bool ok = idx < 32 * FB / 8;
        d_off[j] = ok ? (r * a.HD + f % a.HD + 8 * c) * 2 : -1;
        d_lds[j] = r * DSTR + seg * segw + 8 * c;
    }

    auto load_sub = [&](int64_t t0, u32x4 (&dr)[ND], u32x4 (&yr)[NY]) {
        // dout rows t0..t0+31 of this block's features, y rows t0..t0+31
        const int64_t nt = t_end - t0 < 32 ? t_end - t0 : 32;
        const uint32_t dbytes = nt > 0 ? (uint32_t)nt * a.HD * 2u : 0u;
#pragma unroll
        for (int j = 0; j < ND; ++j) {
            const rsrc_t rd_ = make_buf(d_base[j] + t0 * a.HD * 2, dbytes);
            dr[j] = bload16(rd_, d_off[j] >= 0 ? (uint32_t)d_off[j] : kOOB);
        }
        const rsrc_t ry_ = make_buf((const char *)a.y + t0 * C * 2, nt > 0 ? (uint32_t)nt * C * 2u : 0u);
#pragma unroll
        for (int j = 0; j < NY; ++j) {
            const int idx = tid + j * NT;
            const int r = idx / (C / 8), c8 = idx % (C / 8);
            yr[j] = bload16(ry_, idx < 32 * C / 8 ? (uint32_t)(r * C + c8 * 8) * 2u : kOOB);
        }
    };
    auto store_sub = [&](int buf, const u32x4 (&dr)[ND], const u32x4 (&yr)[NY]) {
#pragma unroll
        for (int j = 0; j < ND; ++j)
            if (d_off[j] >= 0) *(u32x4 *)&dl[buf][d_lds[j]] = dr[j];
#pragma unroll
        for (int j = 0; j < NY; ++j) {
            const int idx = tid + j * NT;
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
    f32x16 acc[TPW], accb = zero16();
#pragma unroll
    for (int j = 0; j < TPW; ++j) acc[j] = zero16();

    const int64_t nsub = (t_end - t_begin + 31) / 32;
    u32x4 dr[NR][ND], yr[NR][NY];
#pragma unroll
    for (int u = 0; u < NR; ++u) load_sub(t_begin + u * 32, dr[u], yr[u]);
    store_sub(0, dr[0], yr[0]);
    load_sub(t_begin + NR * 32, dr[0], yr[0]);
    __syncthreads();
    for (int64_t s0 = 0; s0 < nsub; s0 += NR) {
#pragma unroll
        for (int u = 0; u < NR; ++u) {
            const int64_t sb = s0 + u;
            const int buf = u & 1;
            if (sb < nsub && active) {
                const Tr<bf16_t>::K32 af = load_k32_tr(&dl[buf][ft * 32], DSTR, 0, 32, lane);
#pragma unroll
                for (int j = 0; j < TPW; ++j) {
                    const Tr<bf16_t>::K32 bf = load_k32_tr(&yl[buf][(ct0 + j) * 32], YSTR, 0, 32, lane);
                    Tr<bf16_t>::mma_k32(acc[j], af, bf);
                }
                if (bias_owner) Tr<bf16_t>::mma_k32(accb, af, ones);
            }
            // sub-block sb+1 (loaded NR sub-blocks ago) into the other buffer; its
            // register stage then takes sub-block sb+1+NR
            const int un = (u + 1) % NR;
            store_sub(buf ^ 1, dr[un], yr[un]);
            load_sub(t_begin + (sb + 1 + NR) * 32, dr[un], yr[un]);
            __syncthreads();
        }
    }

    // partial tiles: D[feature ft*32 + sig(rho(i,h))][channel ct*32 + sig(n)]
    if (!active) return;
    const rsrc_t rpw = make_buf(part_w + chunk * (int64_t)F * C, (uint32_t)F * C * 4u);
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
        const int ct = ct0 + j;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int f = f0 + ft * 32 + sig(8 * (i / 4) + 4 * h + (i % 4));
            bstore4(__float_as_uint(acc[j][i]), rpw, (uint32_t)(f * C + ct * 32 + sig(n)) * 4u);
        }
    }
    if (part_b && bias_owner) {
        const rsrc_t rpb = make_buf(part_b + chunk * (int64_t)F, (uint32_t)F * 4u);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int f = f0 + ft * 32 + sig(8 * (i / 4) + 4 * h + (i % 4));
            bstore4(__float_as_uint(accb[i]), rpb, n == 0 ? (uint32_t)f * 4u : kOOB);
        }
    }
}

// out[x] = sum_k part[k][x]: a 256-thread block takes 256 / KS groups of
// four columns and splits k into KS interleaved slices (thread slice ks sums
// k = ks, ks + KS, ... in order); the KS slice sums are then added in slice
// order, so the result does not depend on timing.  Blocks past the first
// array's columns reduce the second array.
template <int KS>
__global__ __launch_bounds__(256) void colsum_kernel(const float *__restrict__ part, int64_t width,
                                                    float *__restrict__ out, const float *__restrict__ part2,
                                                    int64_t width2, float *__restrict__ out2, int64_t n_part) {
    constexpr int QB = 256 / KS;              // four-column groups per block
    __shared__ f32x4 red[KS > 1 ? KS : 1][QB];
    const int ks = threadIdx.x / QB, qb = threadIdx.x % QB;
    int64_t blk = blockIdx.x;
    const int64_t nb1 = (width / 4 + QB - 1) / QB;
    if (blk >= nb1) {
        blk -= nb1;
        part = part2;
        width = width2;
        out = out2;
    }
    const int64_t x4 = (blk * QB + qb) * 4;
    const bool ok = x4 < width;
    const rsrc_t rp = make_buf(part, (uint32_t)(n_part * width * 4));
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
    int64_t k = ks;
    for (; k + 3 * KS < n_part; k += 4 * KS) {
        f32x4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            v[u] = __builtin_bit_cast(f32x4, bload16(rp, ok ? (uint32_t)((k + u * KS) * width + x4) * 4u : kOOB));
#pragma unroll
        for (int u = 0; u < 4; ++u) s += v[u];
    }
    for (; k < n_part; k += KS) s += __builtin_bit_cast(f32x4, bload16(rp, ok ? (uint32_t)(k * width + x4) * 4u : kOOB));
    if constexpr (KS > 1) {
        red[ks][qb] = s;
        __syncthreads();
        if (ks != 0) return;
        s = red[0][qb];
#pragma unroll
        for (int j = 1; j < KS; ++j) s += red[j][qb];
    }
    if (!ok) return;
    const rsrc_t ro = make_buf(out, (uint32_t)(width * 4));
    bstore16(__builtin_bit_cast(u32x4, s), ro, (uint32_t)x4 * 4u);
}

template <int C, int FB>
void launch_dw(dim3 grid, hipStream_t s, const PjBwdArgs &a, int64_t ct, int nfb, int xm, float *pw, float *pb) {
    hipLaunchKernelGGL((dw_kernel<C, FB>), grid, dim3(DwCfg<C, FB>::NT), 0, s, a, ct, nfb, xm, pw, pb);
}

template <int C>
hipError_t launch_c(const PjBwdArgs &a, void *ws, const PjBwdPlan &plan, hipStream_t s) {
    char *w = (char *)ws;
    // without a LayerNorm (a plain linear layer) dY is the input gradient itself
    const bool ln = a.lnw != nullptr;
    void *dy = ln ? w + plan.off_dy : a.dx;
    const int64_t nt = (a.R + 127) / 128;
    // split the channels when the token blocks alone leave CUs idle
    int ncs = 1;
    while (ncs < C / 64 && nt * ncs < 256) ncs *= 2;
    if (C >= 256 && ncs == 4) {
        hipLaunchKernelGGL((dy_kernel<C, C / 4 >= 64 ? C / 4 : 64>), dim3((unsigned)nt, 4), dim3(DyCfg<64>::NT), 0, s,
                           a, dy);
    } else if (C >= 128 && ncs == 2) {
        hipLaunchKernelGGL((dy_kernel<C, C / 2 >= 64 ? C / 2 : 64>), dim3((unsigned)nt, 2),
                           dim3(DyCfg<(C / 2 >= 64 ? C / 2 : 64)>::NT), 0, s, a, dy);
    } else {
        hipLaunchKernelGGL((dy_kernel<C, C>), dim3((unsigned)nt), dim3(DyCfg<C>::NT), 0, s, a, dy);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (ln) {  // LayerNorm backward of dY (bf16) -> dx, dln_w, dln_b
        LnProblem lp{1, C, a.R, 0.0f};
        LnBwdPtrs lx{a.x, a.lnw, a.mean, a.rstd, dy, a.dx, a.dlnw, a.dlnb};
        e = launch_ln_bwd(lp, lx, w + plan.off_ln, s);
        if (e != hipSuccess) return e;
    }
    const int F = a.P * a.HD;
    float *pw = (float *)(w + plan.off_dw);
    float *pb = a.dbias ? (float *)(w + plan.off_db) : nullptr;
    const int fb = proj_bwd_fb(C, a.HD, a.P);
    const int nfb = F / fb;
    const int xcd_map = plan.n_chunks % 8 == 0;
    const dim3 grid((unsigned)(nfb * plan.n_chunks));
    if (fb == 128) {
        launch_dw<C, 128>(grid, s, a, plan.chunk_tokens, nfb, xcd_map, pw, pb);
    } else if (fb == 64) {
        launch_dw<C, 64>(grid, s, a, plan.chunk_tokens, nfb, xcd_map, pw, pb);
    } else {
        launch_dw<C, 32>(grid, s, a, plan.chunk_tokens, nfb, xcd_map, pw, pb);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    // dW and dbias partial sums in one launch (dbias part empty without a
    // bias); the chunk range is split over more threads when there are few
    // columns, so that the launch still has about 256 blocks
    const int64_t wdw = (int64_t)F * C, wdb = a.dbias ? F : 0;
    const int64_t q = wdw / 4;
    if (q >= 65536) {
        hipLaunchKernelGGL((colsum_kernel<1>), dim3((unsigned)((q + 255) / 256 + (wdb / 4 + 255) / 256)), dim3(256), 0,
                           s, pw, wdw, a.dW, pb, wdb, a.dbias, plan.n_chunks);
    } else if (q >= 16384) {
        hipLaunchKernelGGL((colsum_kernel<4>), dim3((unsigned)((q + 63) / 64 + (wdb / 4 + 63) / 64)), dim3(256), 0, s,
                           pw, wdw, a.dW, pb, wdb, a.dbias, plan.n_chunks);
    } else {
        hipLaunchKernelGGL((colsum_kernel<16>), dim3((unsigned)((q + 15) / 16 + (wdb / 4 + 15) / 16)), dim3(256), 0, s,
                           pw, wdw, a.dW, pb, wdb, a.dbias, plan.n_chunks);
    }
    return hipGetLastError();
}

}  // namespace

PjBwdPlan plan_proj_bwd(int64_t R, int C, int HD, int P, bool ln) {
    PjBwdPlan pl{};
    const int F = P * HD;
    const int FB = proj_bwd_fb(C, HD, P);
    const int64_t nfb = F / FB > 0 ? F / FB : 1;
    // about one (feature block, token chunk) workgroup per CU: fewer chunks
    // mean fewer partial sums to write and add up; chunks of whole 32-token
    // sub-blocks
    int64_t nch = (proj_bwd_dw_wgs() + nfb - 1) / nfb;
    // chunks of at least 256 tokens: at few tokens the partial sums would
    // otherwise cost more traffic than the inputs (at 4096 tokens x 256
    // channels, 256-token chunks measured 11.2 us, 512-token chunks 12.8)
    const int64_t nmax = R / 256 > 0 ? R / 256 : 1;
    if (nch > nmax) nch = nmax;
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
    if (ln) off += align256((size_t)R * C * 2);
    pl.off_ln = off;
    if (ln) off += align256(ln_bwd_workspace(lp));
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
