// evo_bwd.hip -- backward kernels of the gated attention with pair bias, gfx950.
//
// Recompute-based backward of o = sigmoid(g) * softmax(s) V with
// s = Q K^T / sqrt(d) + bias + mask (ScaleFold Section 3.3, "Multi Head
// Attention"; the kernel recomputes the probabilities from the saved
// log-sum-exp instead of storing them):
//   dA = dO sigmoid(g),  dG = dO o (1 - sigmoid(g)),  Dsum_i = sum_c dO_ic o_ic
//   P  = exp(s - lse),   dP = dA V^T,   dS = P (dP - Dsum)
//   dV = P^T dA,  dK = dS^T Q / sqrt(d),  dQ = dS K / sqrt(d),
//   dBias[plane] = sum over the plane's rows of dS.
//
// Four kernels:
//   prep   -- elementwise: dA (to workspace), Dsum (to workspace), dG.
//   main   -- one workgroup per (row, head); wave w owns key tile w (32 keys)
//             and loops over the query tiles.  dK and dV of the tile finish
//             in the wave's registers, dQ is summed over the key tiles with
//             LDS float atomics.
//   dbias  -- one workgroup per (bias plane, head, key tile, chunk of rows):
//             recomputes dS for its 32 keys x all queries over the chunk's
//             rows, accumulating in registers, and writes one partial plane
//             tile per chunk.
//   reduce -- sums the partial planes of each (plane, head) into dbias.
// dBias gets its own kernel because a register accumulator for a whole
// (head, L x L) plane does not fit beside the dQ/dK/dV working set; the
// recompute costs two small MFMAs and one exp per logit.  The reduction is a
// fixed-order two-step reduction (register accumulation, then a sum over
// partial planes), so results are bitwise repeatable; global float atomics
// are avoided (they sustain only a few hundred million adds per second on
// this part).
#include <math.h>
#include <stdlib.h>

#include "evo_frag.h"
#include "evo_kernels.h"

namespace evo {

namespace {

constexpr float kLog2e = 1.4426950408889634f;

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// ---------------------------------------------------------------------------
struct PrepArgs {
    const void *out, *dout, *g;
    void *da;      // workspace [N][L][H][D]
    float *dsum;   // workspace [N][H][L]
    void *dg;
    int64_t N, L, srow, stok;
    int H;
};

template <typename T, int D>
__global__ void __launch_bounds__(256) prep_kernel(PrepArgs a) {
    using E = typename Tr<T>::elem;
    constexpr int VEC = Tr<T>::VEC;
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // (r, t, h)
    const int64_t total = a.N * a.L * a.H;
    if (idx >= total) return;
    const int h = (int)(idx % a.H);
    const int64_t rt = idx / a.H;
    const int64_t t = rt % a.L, r = rt / a.L;
    const int64_t tok = r * a.srow + t * a.stok + (int64_t)h * D;
    const E *O = (const E *)a.out + tok;
    const E *dO = (const E *)a.dout + tok;
    const E *G = a.g ? (const E *)a.g + tok : nullptr;
    E *dA = (E *)a.da + idx * D;
    E *dG = a.dg ? (E *)a.dg + tok : nullptr;
    float dsum = 0.0f;
#pragma unroll
    for (int c0 = 0; c0 < D; c0 += VEC) {
        uint4 ov = *reinterpret_cast<const uint4 *>(O + c0);
        uint4 dov = *reinterpret_cast<const uint4 *>(dO + c0);
        uint4 gv = make_uint4(0, 0, 0, 0);
        if (G) gv = *reinterpret_cast<const uint4 *>(G + c0);
        const E *oe = reinterpret_cast<const E *>(&ov);
        const E *de = reinterpret_cast<const E *>(&dov);
        const E *ge = reinterpret_cast<const E *>(&gv);
        uint4 dav, dgv;
        E *dae = reinterpret_cast<E *>(&dav);
        E *dge = reinterpret_cast<E *>(&dgv);
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            const float o = Tr<T>::to_f(oe[e]), d = Tr<T>::to_f(de[e]);
            dsum = __builtin_fmaf(d, o, dsum);
            if (G) {
                const float sg = 1.0f / (1.0f + __builtin_amdgcn_exp2f(-Tr<T>::to_f(ge[e]) * kLog2e));
                dae[e] = Tr<T>::from_f(d * sg);
                dge[e] = Tr<T>::from_f(d * o * (1.0f - sg));
            } else {
                dae[e] = de[e];  // no gate: dA = dO
            }
        }
        *reinterpret_cast<uint4 *>(dA + c0) = dav;
        if (dG) *reinterpret_cast<uint4 *>(dG + c0) = dgv;
    }
    a.dsum[(r * a.H + h) * a.L + t] = dsum;
}

// ---------------------------------------------------------------------------
struct MainArgs {
    const void *q, *k, *v, *bias;
    const uint8_t *mask;
    const float *lse;
    const void *da;
    const float *dsum;
    void *dq, *dk, *dv;
    int64_t L, rpb, srow, stok;
    int H;
    float scale;
};

template <typename T, int D, int NKT>
__global__ void __launch_bounds__(NKT * 64) main_kernel(MainArgs a) {
    using E = typename Tr<T>::elem;
    using K32 = typename Tr<T>::K32;
    constexpr int VEC = Tr<T>::VEC;
    constexpr int LP = NKT * 32;
    constexpr int NT = NKT * 64;
    constexpr int RSTR = D + VEC;    // row-major LDS stride
    constexpr int TSTR = LP + VEC;   // transposed LDS stride
    constexpr int QSTR = D + 1;      // dQ accumulator stride (odd: spreads LDS banks)
    constexpr int SSTR = 32 + VEC;   // dS scratch stride
    __shared__ __attribute__((aligned(16))) E q_lds[LP * RSTR];
    __shared__ __attribute__((aligned(16))) E da_lds[LP * RSTR];
    __shared__ __attribute__((aligned(16))) E qt_lds[D * TSTR];
    __shared__ __attribute__((aligned(16))) E dat_lds[D * TSTR];
    __shared__ __attribute__((aligned(16))) float lse2_lds[LP];
    __shared__ __attribute__((aligned(16))) float dsum_lds[LP];
    __shared__ float dq_acc[LP * QSTR];
    __shared__ __attribute__((aligned(16))) E dsc[NKT * 32 * SSTR];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h2 = lane >> 5, n = lane & 31;
    const int L = (int)a.L;
    // unit -> (row, head), head fastest so the heads of one row run back to
    // back on one XCD
    const int64_t unit = xcd_unit(blockIdx.x, gridDim.x);
    const int hh = (int)(unit % a.H);
    const int64_t r = unit / a.H;
    const int64_t b = r / a.rpb;

    const int kt = wave;
    const int key = kt * 32 + n;
    const int krow_sig = sig(n);                 // permuted operand row of this lane
    const E *bias_plane = a.bias ? (const E *)a.bias + (b * a.H + hh) * (int64_t)L * L : nullptr;

    for (int i = tid; i < LP * QSTR; i += NT) dq_acc[i] = 0.0f;

    {
        const int64_t base = r * a.srow + (int64_t)hh * D;
        // ---- stage Q and dA in both layouts, lse (log2 units) and Dsum
        const E *Q = (const E *)a.q + base;
        const E *dA = (const E *)a.da + ((r * L) * a.H + hh) * D;
        for (int idx = tid; idx < LP * (D / VEC); idx += NT) {
            const int t = idx / (D / VEC), c = (idx % (D / VEC)) * VEC;
            uint4 qv = make_uint4(0, 0, 0, 0), av = make_uint4(0, 0, 0, 0);
            if (t < L) {
                qv = *reinterpret_cast<const uint4 *>(Q + (int64_t)t * a.stok + c);
                av = *reinterpret_cast<const uint4 *>(dA + (int64_t)t * a.H * D + c);
            }
            *reinterpret_cast<uint4 *>(&q_lds[t * RSTR + c]) = qv;
            *reinterpret_cast<uint4 *>(&da_lds[t * RSTR + c]) = av;
            const E *qe = reinterpret_cast<const E *>(&qv);
            const E *ae = reinterpret_cast<const E *>(&av);
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                qt_lds[(c + e) * TSTR + t] = qe[e];
                dat_lds[(c + e) * TSTR + t] = ae[e];
            }
        }
        for (int t = tid; t < LP; t += NT) {
            float l2 = INFINITY, ds = 0.0f;  // padded or fully masked queries: P = 0
            if (t < L) {
                const float l = a.lse[(r * a.H + hh) * a.L + t];
                if (l != -INFINITY) l2 = l * kLog2e;
                ds = a.dsum[(r * a.H + hh) * a.L + t];
            }
            lse2_lds[t] = l2;
            dsum_lds[t] = ds;
        }

        // ---- this wave's key tile: K and V as B operands, K^T as A operand of dQ
        const bool kin = key < L;
        bool kvalid = kin;
        if (kvalid && a.mask) kvalid = a.mask[r * a.L + key] != 0;
        const bool kfull = __ballot(kvalid) == ~0ull;
        const E *K = (const E *)a.k + base;
        const E *V = (const E *)a.v + base;
        ChFrag<T, D> kb, vb;
        if (kin) {
            kb.load(K + (int64_t)key * a.stok, h2);
            vb.load(V + (int64_t)key * a.stok, h2);
        } else {
            kb.zero();
            vb.zero();
        }
        K32 kT;  // kT rows: channel sig(n); k-slots: keys of the tile
        if constexpr (sizeof(E) == 2) {
#pragma unroll
            for (int s = 0; s < 8; ++s) {
                const int j0 = kt * 32 + 8 * h2 + s, j1 = kt * 32 + 16 + 8 * h2 + s;
                uint16_t x0 = 0, x1 = 0;
                if (krow_sig < D && j0 < L) x0 = K[(int64_t)j0 * a.stok + krow_sig];
                if (krow_sig < D && j1 < L) x1 = K[(int64_t)j1 * a.stok + krow_sig];
                kT.v[0][s] = __builtin_bit_cast(__bf16, x0);
                kT.v[1][s] = __builtin_bit_cast(__bf16, x1);
            }
        } else {
#pragma unroll
            for (int u = 0; u < 16; ++u) {
                const int j = kt * 32 + krow(u, h2);
                kT.v[u] = (krow_sig < D && j < L) ? K[(int64_t)j * a.stok + krow_sig] : 0.0f;
            }
        }
        __syncthreads();

        f32x16 dv_acc = zero16(), dk_acc = zero16();
        E *my_dsc = dsc + wave * 32 * SSTR;
        const int nqt = (L + 31) / 32;
#pragma unroll
        for (int qt = 0; qt < NKT; ++qt) {
            if (qt >= nqt) break;
            // S = Q K^T and dP = dA V^T for (32 queries x this wave's 32 keys);
            // lane = key, reg i = query krow(i, h2)
            ChFrag<T, D> qa, daa;
            qa.load(&q_lds[(qt * 32 + krow_sig) * RSTR], h2);
            daa.load(&da_lds[(qt * 32 + krow_sig) * RSTR], h2);
            f32x16 S = zero16(), dP = zero16();
            ChFrag<T, D>::mma(S, qa, kb);
            ChFrag<T, D>::mma(dP, daa, vb);
            float l2[16], dsv[16];
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int q0 = qt * 32 + 16 * half + 8 * h2;
                const float4 *lp = reinterpret_cast<const float4 *>(&lse2_lds[q0]);
                const float4 *dp = reinterpret_cast<const float4 *>(&dsum_lds[q0]);
                float4 x0 = lp[0], x1 = lp[1], y0 = dp[0], y1 = dp[1];
                l2[8 * half + 0] = x0.x; l2[8 * half + 1] = x0.y; l2[8 * half + 2] = x0.z; l2[8 * half + 3] = x0.w;
                l2[8 * half + 4] = x1.x; l2[8 * half + 5] = x1.y; l2[8 * half + 6] = x1.z; l2[8 * half + 7] = x1.w;
                dsv[8 * half + 0] = y0.x; dsv[8 * half + 1] = y0.y; dsv[8 * half + 2] = y0.z; dsv[8 * half + 3] = y0.w;
                dsv[8 * half + 4] = y1.x; dsv[8 * half + 5] = y1.y; dsv[8 * half + 6] = y1.z; dsv[8 * half + 7] = y1.w;
            }
            f32x16 P, dS;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int qi = qt * 32 + krow(i, h2);
                float bv = 0.0f;
                if (bias_plane && kin && qi < L) bv = Tr<T>::to_f(bias_plane[(int64_t)qi * L + key]);
                const float t = __builtin_fmaf(S[i], a.scale, bv);
                float p = __builtin_amdgcn_exp2f(__builtin_fmaf(t, kLog2e, -l2[i]));
                if (!kfull && !kvalid) p = 0.0f;
                P[i] = p;
                dS[i] = p * (dP[i] - dsv[i]);
            }
            const K32 pb = Tr<T>::pack(P);
            const K32 dsb = Tr<T>::pack(dS);
            // dV^T += dA^T P ;  dK^T += Q^T dS   (A rows: channel sig(n))
            K32 dat, qtf;
            if (krow_sig < D) {
                dat = load_k32<T>(&dat_lds[krow_sig * TSTR + qt * 32], h2);
                qtf = load_k32<T>(&qt_lds[krow_sig * TSTR + qt * 32], h2);
            } else {
                dat = zero_k32<T>();
                qtf = zero_k32<T>();
            }
            Tr<T>::mma_k32(dv_acc, dat, pb);
            Tr<T>::mma_k32(dk_acc, qtf, dsb);
            // dQ^T (channels x queries) = K^T dS^T: dS goes through LDS to
            // swap its lane/register roles
#pragma unroll
            for (int i = 0; i < 16; ++i) my_dsc[krow(i, h2) * SSTR + n] = Tr<T>::from_f(dS[i]);
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            const K32 dst = load_k32<T>(&my_dsc[n * SSTR], h2);
            f32x16 dq = zero16();
            Tr<T>::mma_k32(dq, kT, dst);
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int ch = krow(i, h2);
                if (ch < D) atomicAdd(&dq_acc[(qt * 32 + n) * QSTR + ch], dq[i]);
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        }

        // ---- dK and dV of this key tile are complete
        if (kin) {
            E *dKp = (E *)a.dk + base + (int64_t)key * a.stok;
            E *dVp = (E *)a.dv + base + (int64_t)key * a.stok;
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int c0 = 16 * half + 8 * h2;
                if (c0 >= D) continue;
                if constexpr (sizeof(E) == 2) {
                    uint4 wk, wv;
                    uint32_t *pk = reinterpret_cast<uint32_t *>(&wk), *pv = reinterpret_cast<uint32_t *>(&wv);
#pragma unroll
                    for (int s = 0; s < 4; ++s) {
                        pk[s] = (uint32_t)f2bf(dk_acc[8 * half + 2 * s] * a.scale) |
                                ((uint32_t)f2bf(dk_acc[8 * half + 2 * s + 1] * a.scale) << 16);
                        pv[s] = (uint32_t)f2bf(dv_acc[8 * half + 2 * s]) |
                                ((uint32_t)f2bf(dv_acc[8 * half + 2 * s + 1]) << 16);
                    }
                    *reinterpret_cast<uint4 *>(dKp + c0) = wk;
                    *reinterpret_cast<uint4 *>(dVp + c0) = wv;
                } else {
                    const int o = 8 * half;
                    *reinterpret_cast<float4 *>(dKp + c0) =
                        make_float4(dk_acc[o] * a.scale, dk_acc[o + 1] * a.scale, dk_acc[o + 2] * a.scale, dk_acc[o + 3] * a.scale);
                    *reinterpret_cast<float4 *>(dKp + c0 + 4) =
                        make_float4(dk_acc[o + 4] * a.scale, dk_acc[o + 5] * a.scale, dk_acc[o + 6] * a.scale, dk_acc[o + 7] * a.scale);
                    *reinterpret_cast<float4 *>(dVp + c0) = make_float4(dv_acc[o], dv_acc[o + 1], dv_acc[o + 2], dv_acc[o + 3]);
                    *reinterpret_cast<float4 *>(dVp + c0 + 4) = make_float4(dv_acc[o + 4], dv_acc[o + 5], dv_acc[o + 6], dv_acc[o + 7]);
                }
            }
        }
        __syncthreads();  // every wave's dQ contributions are in dq_acc
        E *dQ = (E *)a.dq + base;
        for (int idx = tid; idx < L * D; idx += NT) {
            const int t = idx / D, c = idx % D;
            dQ[(int64_t)t * a.stok + c] = Tr<T>::from_f(dq_acc[t * QSTR + c] * a.scale);
        }
    }
}

// ---------------------------------------------------------------------------
struct DbiasArgs {
    const void *q, *k, *v, *bias;
    const uint8_t *mask;
    const float *lse;
    const void *da;
    const float *dsum;
    float *part;   // [B][H][chunks][L][L]
    int64_t L, rpb, srow, stok, chunks, rows_per_chunk;
    int H;
    float scale;
};

// One workgroup = (plane b, head h, key tile kt, chunk of rows).  Wave w owns
// query tiles w, w+4, ...; lane = key, registers = queries (same D layout as
// the main kernel), so the accumulator is NQW x 16 registers per lane.
template <typename T, int D, int NKT>
__global__ void __launch_bounds__(256) dbias_kernel(DbiasArgs a) {
    using E = typename Tr<T>::elem;
    constexpr int NQW = (NKT + 3) / 4;  // query tiles per wave
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h2 = lane >> 5, n = lane & 31;
    const int L = (int)a.L;
    const int nkt = (L + 31) / 32;
    // unit -> (b, chunk, kt, head), head fastest
    const int64_t unit = xcd_unit(blockIdx.x, gridDim.x);
    const int hh = (int)(unit % a.H);
    int64_t rest = unit / a.H;
    const int kt = (int)(rest % nkt);
    rest /= nkt;
    const int64_t chunk = rest % a.chunks, b = rest / a.chunks;
    const int64_t r_begin = b * a.rpb + chunk * a.rows_per_chunk;
    int64_t r_end = r_begin + a.rows_per_chunk;
    if (r_end > (b + 1) * a.rpb) r_end = (b + 1) * a.rpb;

    const int key = kt * 32 + n;
    const bool kin = key < L;
    const int krow_sig = sig(n);
    const E *bias_plane = (const E *)a.bias + (b * a.H + hh) * (int64_t)L * L;

    // bias tile (constant over rows) and accumulators
    float bt[NQW][16];
    f32x16 acc[NQW];
#pragma unroll
    for (int j = 0; j < NQW; ++j) {
        acc[j] = zero16();
        const int qt = wave + 4 * j;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int qi = qt * 32 + krow(i, h2);
            bt[j][i] = (kin && qi < L) ? Tr<T>::to_f(bias_plane[(int64_t)qi * L + key]) : 0.0f;
        }
    }

    for (int64_t r = r_begin; r < r_end; ++r) {
        const int64_t base = r * a.srow + (int64_t)hh * D;
        bool kvalid = kin;
        if (kvalid && a.mask) kvalid = a.mask[r * a.L + key] != 0;
        if (__ballot(kvalid) == 0ull) continue;  // every key of the tile masked: dS = 0
        const bool kfull = __ballot(kvalid) == ~0ull;
        const E *K = (const E *)a.k + base;
        const E *V = (const E *)a.v + base;
        ChFrag<T, D> kb, vb;
        if (kin) {
            kb.load(K + (int64_t)key * a.stok, h2);
            vb.load(V + (int64_t)key * a.stok, h2);
        } else {
            kb.zero();
            vb.zero();
        }
        const E *Q = (const E *)a.q + base;
        const E *dA = (const E *)a.da + ((r * L) * a.H + hh) * D;
        const float *lse = a.lse + (r * a.H + hh) * a.L;
        const float *dsum = a.dsum + (r * a.H + hh) * a.L;
#pragma unroll
        for (int j = 0; j < NQW; ++j) {
            const int qt = wave + 4 * j;
            if (qt * 32 >= L) break;
            const int qrow = qt * 32 + krow_sig;  // A-operand row of this lane
            ChFrag<T, D> qa, daa;
            if (qrow < L) {
                qa.load(Q + (int64_t)qrow * a.stok, h2);
                daa.load(dA + (int64_t)qrow * a.H * D, h2);
            } else {
                qa.zero();
                daa.zero();
            }
            f32x16 S = zero16(), dP = zero16();
            ChFrag<T, D>::mma(S, qa, kb);
            ChFrag<T, D>::mma(dP, daa, vb);
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int qi = qt * 32 + krow(i, h2);
                float l2 = INFINITY, ds = 0.0f;
                if (qi < L) {
                    const float l = lse[qi];
                    if (l != -INFINITY) l2 = l * kLog2e;
                    ds = dsum[qi];
                }
                const float t = __builtin_fmaf(S[i], a.scale, bt[j][i]);
                float p = __builtin_amdgcn_exp2f(__builtin_fmaf(t, kLog2e, -l2));
                if (!kfull && !kvalid) p = 0.0f;
                acc[j][i] += p * (dP[i] - ds);
            }
        }
    }

    if (kin) {
        float *pp = a.part + ((b * a.H + hh) * a.chunks + chunk) * (int64_t)L * L;
#pragma unroll
        for (int j = 0; j < NQW; ++j) {
            const int qt = wave + 4 * j;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int qi = qt * 32 + krow(i, h2);
                if (qi < L) pp[(int64_t)qi * L + key] = acc[j][i];
            }
        }
    }
}

// dbias[p][x] = sum over chunks c of part[p][c][x], in chunk order
__global__ void __launch_bounds__(256) dbias_reduce_kernel(const float *__restrict__ part, float *__restrict__ dbias,
                                                        int64_t planes /* B*H */, int64_t chunks, int64_t plane_elems) {
    const int64_t total = planes * plane_elems;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t p = e / plane_elems, x = e % plane_elems;
        const float *src = part + p * chunks * plane_elems + x;
        float acc = 0.0f;
        for (int64_t c = 0; c < chunks; ++c) acc += src[c * plane_elems];
        dbias[e] = acc;
    }
}

// ---------------------------------------------------------------------------
template <typename T, int D>
hipError_t launch_prep(const Problem &p, const PrepArgs &pa, hipStream_t s) {
    const int64_t total = p.N * p.L * p.H;
    const int64_t blocks = (total + 255) / 256;
    hipLaunchKernelGGL((prep_kernel<T, D>), dim3((unsigned)blocks), dim3(256), 0, s, pa);
    return hipGetLastError();
}

template <typename T, int D, int NKT>
hipError_t launch_main_dbias(const Problem &p, const MainArgs &ma, const DbiasArgs &da, const BwdPlan &plan,
                             hipStream_t s) {
    hipLaunchKernelGGL((main_kernel<T, D, NKT>), dim3((unsigned)(p.N * p.H)), dim3(NKT * 64), 0, s, ma);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !da.bias) return e;
    hipLaunchKernelGGL((dbias_kernel<T, D, NKT>), dim3((unsigned)plan.n_wg), dim3(256), 0, s, da);
    return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_main_d(const Problem &p, const MainArgs &ma, const DbiasArgs &da, const BwdPlan &plan,
                         hipStream_t s) {
    const int64_t nkt = (p.L + 31) / 32;
    if (nkt <= 1) return launch_main_dbias<T, D, 1>(p, ma, da, plan, s);
    if (nkt <= 2) return launch_main_dbias<T, D, 2>(p, ma, da, plan, s);
    if (nkt <= 4) return launch_main_dbias<T, D, 4>(p, ma, da, plan, s);
    if constexpr (sizeof(typename Tr<T>::elem) == 4 && D == 32) {
        return hipErrorInvalidValue;  // rejected by the ABI layer before any launch
    } else {
        return launch_main_dbias<T, D, 8>(p, ma, da, plan, s);
    }
}

template <typename T>
hipError_t launch_bwd_t(const Problem &p, const BwdPtrs &x, void *ws, const BwdPlan &plan, hipStream_t s) {
    char *w = (char *)ws;
    PrepArgs pa;
    pa.out = x.out; pa.dout = x.dout; pa.g = x.g;
    pa.da = w + plan.off_da;
    pa.dsum = (float *)(w + plan.off_dsum);
    pa.dg = x.dg;
    pa.N = p.N; pa.L = p.L; pa.srow = p.srow; pa.stok = p.stok; pa.H = p.H;
    hipError_t e;
    switch (p.D) {
        case 8: e = launch_prep<T, 8>(p, pa, s); break;
        case 16: e = launch_prep<T, 16>(p, pa, s); break;
        default: e = launch_prep<T, 32>(p, pa, s); break;
    }
    if (e != hipSuccess) return e;

    const int64_t rpb = x.bias ? p.rpb : p.N;
    const float scale = 1.0f / sqrtf((float)p.D);
    MainArgs ma;
    ma.q = x.q; ma.k = x.k; ma.v = x.v; ma.bias = x.bias; ma.mask = x.mask; ma.lse = x.lse;
    ma.da = pa.da; ma.dsum = pa.dsum;
    ma.dq = x.dq; ma.dk = x.dk; ma.dv = x.dv;
    ma.L = p.L; ma.rpb = rpb; ma.srow = p.srow; ma.stok = p.stok; ma.H = p.H; ma.scale = scale;
    DbiasArgs da;
    da.q = x.q; da.k = x.k; da.v = x.v; da.bias = x.bias; da.mask = x.mask; da.lse = x.lse;
    da.da = pa.da; da.dsum = pa.dsum;
    da.part = (float *)(w + plan.off_part);
    da.L = p.L; da.rpb = rpb; da.srow = p.srow; da.stok = p.stok;
    da.chunks = plan.chunks; da.rows_per_chunk = plan.rows_per_chunk;
    da.H = p.H; da.scale = scale;
    switch (p.D) {
        case 8: e = launch_main_d<T, 8>(p, ma, da, plan, s); break;
        case 16: e = launch_main_d<T, 16>(p, ma, da, plan, s); break;
        default: e = launch_main_d<T, 32>(p, ma, da, plan, s); break;
    }
    if (e != hipSuccess || !x.bias) return e;

    const int64_t planes = (p.N / p.rpb) * p.H;
    const int64_t pe = p.L * p.L;
    int64_t blocks = (planes * pe + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(dbias_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                       (const float *)(w + plan.off_part), x.dbias, planes, plan.chunks, pe);
    return hipGetLastError();
}

}  // namespace

BwdPlan plan_bwd(const Problem &p, bool has_bias) {
    BwdPlan pl;
    const int64_t es = p.dtype == 1 ? 2 : 4;
    const int64_t planes = has_bias ? p.N / p.rpb : 0;
    const int64_t nkt = (p.L + 31) / 32;
    int64_t target = 1024;  // dbias workgroups (4 waves each) to fill 256 CUs
    if (const char *env = getenv("EVO_ATTN_DBIAS_WG")) {
        const long v = atol(env);
        if (v > 0) target = v;
    }
    int64_t chunks = 0, g = 1;
    if (has_bias && p.rpb > 0 && nkt > 0) {
        const int64_t base = planes * p.H * nkt;
        chunks = (target + base - 1) / base;
        if (chunks < 1) chunks = 1;
        if (chunks > p.rpb) chunks = p.rpb;
        g = (p.rpb + chunks - 1) / chunks;
        chunks = (p.rpb + g - 1) / g;
    }
    pl.chunks = chunks;
    pl.rows_per_chunk = g;
    pl.n_wg = planes * p.H * nkt * chunks;
    size_t off = 0;
    pl.off_da = off;
    off = align256(off + (size_t)(p.N * p.L * p.H * p.D * es));
    pl.off_dsum = off;
    off = align256(off + (size_t)(p.N * p.H * p.L) * 4);
    pl.off_part = off;
    if (has_bias) off = align256(off + (size_t)(planes * p.H * chunks * p.L * p.L) * 4);
    pl.total = off;
    return pl;
}

hipError_t launch_bwd(const Problem &p, const BwdPtrs &x, void *ws, const BwdPlan &plan, hipStream_t s) {
    if (p.dtype == 1) return launch_bwd_t<bf16_t>(p, x, ws, plan, s);
    return launch_bwd_t<float>(p, x, ws, plan, s);
}

}  // namespace evo
