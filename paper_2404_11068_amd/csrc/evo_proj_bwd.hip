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

// features per workgroup of the weight-gradient pass: a block never spans two
// projections (it divides HD); 128 when the channel tiles alone would leave
// waves idle (C = 64)
inline int proj_bwd_dw_wgs() {
    static const int v = [] {
        const char *e = getenv("EVO_PROJ_DW_WGS");
        const int x = e ? atoi(e) : 0;
        return x >= 8 && x <= 65536 ? x : 256;
    }();
    return v;
}

inline int proj_bwd_fb(int C, int HD) {
    if (C == 64 && HD % 128 == 0) return 128;
    return HD % 64 == 0 ? 64 : 32;
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
// dY tile of 128 tokens x C channels.  Output tiles (token block tb, channel
// tile ct): wave w takes tb = w % 4 and channel tiles ct = w / 4 + 2 j.  The
// contraction runs over stages of 64 features.  Each wave reads its dout
// fragments straight from global memory into a ring of four register stages
// (issued four stages before use, so the HBM latency overlaps the products of
// the stages in between); the weight stage goes through LDS, double-buffered,
// its global loads issued two stages ahead.
template <int C>
__global__ __launch_bounds__(64 * kPbwWaves) void dy_kernel(PjBwdArgs a, void *__restrict__ dy) {
    constexpr int TM = 128, KC = 64, NR = 4;
    constexpr int NCT = C / 32;               // channel tiles
    constexpr int TPW = NCT / 2;              // channel tiles per wave: cg + 2 j < NCT
    static_assert(NCT >= 2 && NCT % 2 == 0, "dy_kernel takes C = 64, 128, 256");
    constexpr int WSTR = C + kLdsPad;         // LDS row stride of a weight stage (elements)
    constexpr int NWL = (KC * C / 8 + 64 * kPbwWaves - 1) / (64 * kPbwWaves);  // 16-byte loads per thread
    constexpr int OSTR = 40;                  // staging row stride (elements) of a 32x32 output tile
    constexpr int LW = 2 * KC * WSTR, LS = kPbwWaves * 32 * OSTR;
    __shared__ __attribute__((aligned(16))) uint16_t lds[LW > LS ? LW : LS];
    uint16_t *wl0 = lds, *wl1 = lds + KC * WSTR;
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

    // dout rows of this token block.  The k32 steps (32 features, inside one
    // projection) are loaded in order, two per stage: `cur` is the projection
    // being read at feature offset lfl, `nx1..nx3` the ones after it (past the
    // last projection the resource is empty and its loads read zeros).  All of
    // it stays in scalar registers: a per-lane copy would turn every load into
    // a loop over distinct resources.
    const uint32_t ablk = (uint32_t)nrows * a.HD * 2u;
    const int64_t aoff = row0 * a.HD * 2;
    const char *cur = (const char *)a.dout0 + aoff, *nx1 = (const char *)a.dout1 + aoff;
    const char *nx2 = (const char *)a.dout2 + aoff, *nx3 = (const char *)a.dout3 + aoff;
    const uint32_t arow = (uint32_t)(tb * 32 + n) * a.HD * 2u + 16u * h;
    int lp = 0, lfl = 0;
    auto load_a = [&](u32x4 (&r)[4]) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const rsrc_t ro = make_buf(cur, __builtin_amdgcn_readfirstlane(lp < a.P ? ablk : 0u));
            const uint32_t off = arow + (uint32_t)lfl * 2u;
            r[2 * t] = bload16(ro, off);
            r[2 * t + 1] = bload16(ro, off + 32u);
            lfl += 32;
            const bool wrap = lfl == a.HD;
            lfl = __builtin_amdgcn_readfirstlane(wrap ? 0 : lfl);
            lp = __builtin_amdgcn_readfirstlane(wrap ? lp + 1 : lp);
            cur = uniform_ptr(wrap ? nx1 : cur);
            nx1 = uniform_ptr(wrap ? nx2 : nx1);
            nx2 = uniform_ptr(wrap ? nx3 : nx2);
        }
    };
    // weight rows s*KC .. s*KC+KC-1 (rows past F read as zeros)
    auto load_w = [&](int s, u32x4 (&r)[NWL]) {
#pragma unroll
        for (int j = 0; j < NWL; ++j) {
            const int idx = tid + j * 64 * kPbwWaves;
            const int rr = idx / (C / 8), c8 = idx % (C / 8);
            r[j] = bload16(rW, idx < KC * C / 8 ? (uint32_t)((s * KC + rr) * C + c8 * 8) * 2u : kOOB);
        }
    };
    auto store_w = [&](uint16_t *wl, const u32x4 (&r)[NWL]) {
#pragma unroll
        for (int j = 0; j < NWL; ++j) {
            const int idx = tid + j * 64 * kPbwWaves;
            if (idx < KC * C / 8) {
                const int rr = idx / (C / 8), c8 = idx % (C / 8);
                *(u32x4 *)&wl[rr * WSTR + c8 * 8] = r[j];
            }
        }
    };

    // Loads form one in-order stream (the memory counter retires them in
    // issue order, so a wait for one load is a wait for every older one): in
    // each stage, dout of stage s + NR, then the weight rows of stage
    // s + NR + 1; stage s then consumes its dout and the weight rows of s + 1,
    // both issued NR stages earlier.
    f32x16 acc[TPW];
#pragma unroll
    for (int j = 0; j < TPW; ++j) acc[j] = zero16();
    u32x4 ar[NR][4], wr[NR][NWL];
    load_w(0, wr[0]);
#pragma unroll
    for (int u = 0; u < NR; ++u) {
        load_a(ar[u]);
        if (u + 1 < NR) load_w(u + 1, wr[u + 1]);
    }
    store_w(wl0, wr[0]);
    load_w(NR, wr[0]);
    __syncthreads();
    for (int s0 = 0; s0 < NS; s0 += NR) {
#pragma unroll
        for (int u = 0; u < NR; ++u) {
            const int s = s0 + u;
            const uint16_t *wl = (u & 1) ? wl1 : wl0;
            if (s < NS) {
#pragma unroll
                for (int t = 0; t < 2; ++t) {
                    Tr<bf16_t>::K32 af;
                    af.v[0] = __builtin_bit_cast(bf16x8, ar[u][2 * t]);
                    af.v[1] = __builtin_bit_cast(bf16x8, ar[u][2 * t + 1]);
#pragma unroll
                    for (int j = 0; j < TPW; ++j) {
                        const Tr<bf16_t>::K32 bf = load_k32_tr(&wl[(cg + 2 * j) * 32], WSTR, 32 * t, 32, lane);
                        Tr<bf16_t>::mma_k32(acc[j], af, bf);
                    }
                }
            }
            const int un = (u + 1) % NR;
            store_w((u & 1) ? wl0 : wl1, wr[un]);  // weight rows of stage s + 1
            load_a(ar[u]);                         // dout of stage s + NR
            load_w(s + NR + 1, wr[un]);
            __syncthreads();
        }
    }

    // epilogue: D[token rho(i,h)][channel ct*32 + sig(n)] -> bf16 -> token rows
    const rsrc_t rd = make_buf((char *)dy + row0 * C * 2, (uint32_t)nrows * C * 2);
    uint16_t *st = lds + wave * 32 * OSTR;
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
        const int ct = cg + 2 * j;
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
// double-buffered); their global loads run through a ring of four register
// stages, issued four sub-blocks before the sub-block is staged.  Wave w owns
// TPW consecutive output tiles of the (FB/32) x (C/32) grid, all in one
// feature tile, so its dout fragment serves all of them.  One wave per
// feature tile (spread over the SIMDs) also sums dbias through an all-ones
// operand.  With `xcd_map`, the feature blocks of one token chunk are placed
// on one XCD (workgroups are dealt to the eight XCDs in turn), so that
// chunk's y rows are fetched into that XCD's L2 once.
template <int C, int FB>
__global__ __launch_bounds__(64 * kPbwWaves) void dw_kernel(PjBwdArgs a, int64_t chunk_tokens, int nfb, int xcd_map,
                                                          float *__restrict__ part_w, float *__restrict__ part_b) {
    constexpr int NFT = FB / 32, NCT = C / 32, NT = NFT * NCT;
    constexpr int TPW = NT / kPbwWaves > 0 ? NT / kPbwWaves : 1;
    constexpr int WPF = NCT / TPW;            // waves per feature tile
    constexpr int NR = 4;
    constexpr int DSTR = FB + kLdsPad, YSTR = C + kLdsPad;
    constexpr int ND = (32 * FB / 8 + 64 * kPbwWaves - 1) / (64 * kPbwWaves);
    constexpr int NY = (32 * C / 8 + 64 * kPbwWaves - 1) / (64 * kPbwWaves);
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
    // the feature block lies inside one projection (HD is a multiple of FB)
    const int p = f0 / a.HD, fl0 = f0 % a.HD;
    const int ft = wave / WPF, ct0 = (wave % WPF) * TPW;
    const bool active = ft < NFT;
    const bool bias_owner = active && (wave % WPF) == ft % WPF;

    auto load_sub = [&](int64_t t0, u32x4 (&dr)[ND], u32x4 (&yr)[NY]) {
        // dout rows t0..t0+31 of this projection's features fl0..fl0+FB, y rows t0..t0+31
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
    auto store_sub = [&](int buf, const u32x4 (&dr)[ND], const u32x4 (&yr)[NY]) {
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

// out[x] = sum_k part[k][x] in k order, four columns per thread; the threads
// past the first array's columns reduce the second array
__global__ __launch_bounds__(256) void colsum_kernel(const float *__restrict__ part, int64_t width,
                                                    float *__restrict__ out, const float *__restrict__ part2,
                                                    int64_t width2, float *__restrict__ out2, int64_t n_part) {
    int64_t x4 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
    const int64_t w1 = (width + 1023) / 1024 * 1024;  // first array's threads end on a block boundary
    if (x4 >= w1) {
        x4 -= w1;
        part = part2;
        width = width2;
        out = out2;
    }
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

template <int C, int FB>
void launch_dw(dim3 grid, hipStream_t s, const PjBwdArgs &a, int64_t ct, int nfb, int xm, float *pw, float *pb) {
    hipLaunchKernelGGL((dw_kernel<C, FB>), grid, dim3(64 * kPbwWaves), 0, s, a, ct, nfb, xm, pw, pb);
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
    // dW and dbias partial sums in one launch (dbias part empty without a bias)
    const int64_t wdw = (int64_t)F * C, wdb = a.dbias ? F : 0;
    const int64_t nblk = (wdw + 1023) / 1024 + (wdb + 1023) / 1024;
    hipLaunchKernelGGL(colsum_kernel, dim3((unsigned)nblk), dim3(256), 0, s, pw, wdw, a.dW, pb, wdb, a.dbias,
                       plan.n_chunks);
    return hipGetLastError();
}

}  // namespace

PjBwdPlan plan_proj_bwd(int64_t R, int C, int HD, int P) {
    PjBwdPlan pl{};
    const int F = P * HD;
    const int FB = proj_bwd_fb(C, HD);
    const int64_t nfb = F / FB > 0 ? F / FB : 1;
    // about one (feature block, token chunk) workgroup per CU: fewer chunks
    // mean fewer partial sums to write and add up; chunks of whole 32-token
    // sub-blocks
    int64_t nch = (proj_bwd_dw_wgs() + nfb - 1) / nfb;
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
