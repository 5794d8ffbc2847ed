// evo_bwd.hip -- backward kernels of the gated attention with pair bias, gfx950.
//
// Recompute-based backward of o = sigmoid(g) * softmax(s) V with
// s = Q K^T / sqrt(d) + bias + mask (ScaleFold Section 3.3, "Multi Head
// Attention"; the probabilities are recomputed from the saved log-sum-exp):
//   dA = dO sigmoid(g),  dG = dO o (1 - sigmoid(g)),  Dsum_i = sum_c dO_ic o_ic
//   P  = exp(s - lse),   dP = dA V^T,   dS = P (dP - Dsum)
//   dV = P^T dA,  dK = dS^T Q / sqrt(d),  dQ = dS K / sqrt(d),
//   dBias[plane] = sum over the plane's rows of dS.
//
// dK and dV are sums over queries, dQ a sum over keys and dBias a sum over
// rows.  No single tiling finishes all three in registers, and global or LDS
// float atomics are slow on this part (a few hundred million adds per
// second; LDS atomics left a first version of this kernel waiting on LDS
// half of the time), so the work is split into two passes that each
// recompute P and dS in the orientation their sums need:
//
//   kv      one workgroup per (row, head); wave w owns key tile w (32 keys),
//           lane = key, registers = queries.  dK and dV finish in registers.
//           It also does the elementwise part (dA, Dsum, dG) while staging,
//           and leaves dA and Dsum in the workspace for the second pass.
//   qbias   one workgroup per (bias plane, head, 32-query tile, chunk of
//           rows); wave w owns key tile w, lane = query, registers = keys.
//           dQ is summed over the waves through LDS in a fixed order; dS is
//           accumulated over the chunk's rows in registers and written once
//           per chunk as a partial dBias tile.
//   reduce  sums the partial dBias planes in chunk order.
// Every sum has a fixed order, so all outputs are bitwise repeatable.
#include <math.h>
#include <stdlib.h>

#include "evo_frag.h"
#include "evo_kernels.h"

namespace evo {

namespace {

constexpr float kLog2e = 1.4426950408889634f;

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// 8 consecutive values row[j0 .. j0+7] as fp32; entries at or beyond n read as 0
template <typename T>
__device__ __forceinline__ void load_row8(const typename Tr<T>::elem *row, int j0, int n, bool vec_ok,
                                          float *out8) {
    using E = typename Tr<T>::elem;
    if (vec_ok && j0 + 8 <= n) {
        if constexpr (sizeof(E) == 2) {
            uint4 u = *reinterpret_cast<const uint4 *>(row + j0);
            uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                out8[2 * s] = __builtin_bit_cast(float, w[s] << 16);
                out8[2 * s + 1] = __builtin_bit_cast(float, w[s] & 0xffff0000u);
            }
        } else {
            float4 a = *reinterpret_cast<const float4 *>(row + j0);
            float4 b = *reinterpret_cast<const float4 *>(row + j0 + 4);
            out8[0] = a.x; out8[1] = a.y; out8[2] = a.z; out8[3] = a.w;
            out8[4] = b.x; out8[5] = b.y; out8[6] = b.z; out8[7] = b.w;
        }
    } else {
#pragma unroll
        for (int s = 0; s < 8; ++s) out8[s] = (j0 + s < n) ? Tr<T>::to_f(row[j0 + s]) : 0.0f;
    }
}

// ---------------------------------------------------------------------------
// biasT[p][j][i] = bias[p][i][j] for every (plane, head) p; 32x32 tiles via LDS
template <typename E>
__global__ void __launch_bounds__(256) transpose_kernel(const E *__restrict__ src, E *__restrict__ dst, int64_t L,
                                                     int64_t tiles) {
    __shared__ E tile[32][33];
    const int64_t blk = blockIdx.x;
    const int64_t p = blk / (tiles * tiles);
    const int64_t tij = blk % (tiles * tiles);
    const int64_t i0 = (tij / tiles) * 32, j0 = (tij % tiles) * 32;
    const E *s = src + p * L * L;
    E *d = dst + p * L * L;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    for (int k = ty; k < 32; k += 8) {
        const int64_t i = i0 + k, j = j0 + tx;
        if (i < L && j < L) tile[k][tx] = s[i * L + j];
    }
    __syncthreads();
    for (int k = ty; k < 32; k += 8) {
        const int64_t j = j0 + k, i = i0 + tx;
        if (i < L && j < L) d[j * L + i] = tile[tx][k];
    }
}

// ---------------------------------------------------------------------------
struct KvArgs {
    const void *q, *k, *v, *g, *out, *dout, *biasT;
    const uint8_t *mask;
    const float *lse;
    void *dk, *dv, *dg;
    void *da;     // workspace [N][H][L][D]
    float *dsum;  // workspace [N][H][L]
    int64_t L, rpb, srow, stok;
    int H;
    float scale;
};

template <typename T, int D, int NKT>
__global__ void __launch_bounds__(NKT * 64) kv_kernel(KvArgs a) {
    using E = typename Tr<T>::elem;
    using K32 = typename Tr<T>::K32;
    constexpr int VEC = Tr<T>::VEC;
    constexpr int CPT = D / VEC;     // 16-byte chunks per token
    constexpr int LP = NKT * 32;
    constexpr int NT = NKT * 64;
    constexpr int RSTR = D + VEC;    // row-major LDS stride
    constexpr int TSTR = LP + VEC;   // transposed LDS stride
    // bf16: Q^T and dA^T fragments come from the transposing LDS read of the
    // row-major tiles; fp32 keeps explicit transposed copies
    constexpr bool kTr = sizeof(E) == 2;
    __shared__ __attribute__((aligned(16))) E q_lds[LP * RSTR];
    __shared__ __attribute__((aligned(16))) E da_lds[LP * RSTR];
    __shared__ __attribute__((aligned(16))) E qt_lds[kTr ? 8 : D * TSTR];
    __shared__ __attribute__((aligned(16))) E dat_lds[kTr ? 8 : D * TSTR];
    __shared__ __attribute__((aligned(16))) float lse2_lds[LP];
    __shared__ __attribute__((aligned(16))) float dsum_lds[LP];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h2 = lane >> 5, n = lane & 31;
    const int L = (int)a.L;
    const int64_t unit = xcd_unit(blockIdx.x, gridDim.x);  // (row, head), head fastest
    const int hh = (int)(unit % a.H);
    const int64_t r = unit / a.H;
    const int64_t b = r / a.rpb;
    const int64_t base = r * a.srow + (int64_t)hh * D;
    const int64_t rh = r * a.H + hh;

    // ---- stage Q and dA (both layouts); dA, Dsum and dG come from dO, O, G here
    {
        const E *Q = (const E *)a.q + base;
        const E *O = (const E *)a.out + base;
        const E *dO = (const E *)a.dout + base;
        const E *G = a.g ? (const E *)a.g + base : nullptr;
        E *dG = a.dg ? (E *)a.dg + base : nullptr;
        E *dAw = (E *)a.da + rh * (int64_t)L * D;
        for (int idx = tid; idx < LP * CPT; idx += NT) {
            const int t = idx / CPT, c = (idx % CPT) * VEC;
            const bool valid = t < L;
            uint4 qv = make_uint4(0, 0, 0, 0), ov = qv, dov = qv, gv = qv;
            if (valid) {
                const int64_t off = (int64_t)t * a.stok + c;
                qv = *reinterpret_cast<const uint4 *>(Q + off);
                ov = *reinterpret_cast<const uint4 *>(O + off);
                dov = *reinterpret_cast<const uint4 *>(dO + off);
                if (G) gv = *reinterpret_cast<const uint4 *>(G + off);
            }
            const E *oe = reinterpret_cast<const E *>(&ov);
            const E *de = reinterpret_cast<const E *>(&dov);
            const E *ge = reinterpret_cast<const E *>(&gv);
            uint4 dav, dgv;
            E *dae = reinterpret_cast<E *>(&dav);
            E *dge = reinterpret_cast<E *>(&dgv);
            float part = 0.0f;
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                const float o = Tr<T>::to_f(oe[e]), d = Tr<T>::to_f(de[e]);
                part = __builtin_fmaf(d, o, part);
                if (G) {
                    const float sg = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-Tr<T>::to_f(ge[e]) * kLog2e));
                    dae[e] = Tr<T>::from_f(d * sg);
                    dge[e] = Tr<T>::from_f(d * o * (1.0f - sg));
                } else {
                    dae[e] = de[e];
                }
            }
            // Dsum of the token: sum over its CPT consecutive lanes
#pragma unroll
            for (int off = 1; off < CPT; off <<= 1) part += __shfl_xor(part, off);
            if (valid) {
                if (dG) *reinterpret_cast<uint4 *>(dG + (int64_t)t * a.stok + c) = dgv;
                *reinterpret_cast<uint4 *>(dAw + (int64_t)t * D + c) = dav;
                if (c == 0) a.dsum[rh * L + t] = part;
            }
            if (c == 0) dsum_lds[t] = valid ? part : 0.0f;
            *reinterpret_cast<uint4 *>(&q_lds[t * RSTR + c]) = qv;
            *reinterpret_cast<uint4 *>(&da_lds[t * RSTR + c]) = dav;
            if constexpr (!kTr) {
                const E *qe = reinterpret_cast<const E *>(&qv);
#pragma unroll
                for (int e = 0; e < VEC; ++e) {
                    qt_lds[(c + e) * TSTR + t] = qe[e];
                    dat_lds[(c + e) * TSTR + t] = dae[e];
                }
            }
        }
        for (int t = tid; t < LP; t += NT) {
            float l2 = INFINITY;  // padded or fully masked queries: P = 0
            if (t < L) {
                const float l = a.lse[rh * L + t];
                if (l != -INFINITY) l2 = l * kLog2e;
            }
            lse2_lds[t] = l2;
        }
    }

    // ---- this wave's key tile: K and V as B operands (lane = key)
    const int kt = wave;
    const int key = kt * 32 + n;
    const int arow = sig(n);  // permuted A-operand row of this lane
    const bool kin = key < L;
    bool kvalid = kin;
    if (kvalid && a.mask) kvalid = a.mask[r * a.L + key] != 0;
    const bool kfull = __ballot(kvalid) == ~0ull;
    ChFrag<T, D> kb, vb;
    if (kin) {
        kb.load((const E *)a.k + base + (int64_t)key * a.stok, h2);
        vb.load((const E *)a.v + base + (int64_t)key * a.stok, h2);
    } else {
        kb.zero();
        vb.zero();
    }
    const E *brow = a.biasT ? (const E *)a.biasT + ((b * a.H + hh) * (int64_t)L + (kin ? key : 0)) * L : nullptr;
    const bool bias_vec = (L % VEC) == 0;
    __syncthreads();

    f32x16 dv_acc = zero16(), dk_acc = zero16();
    const int nqt = (L + 31) / 32;
#pragma unroll
    for (int qt = 0; qt < NKT; ++qt) {
        if (qt >= nqt) break;
        // S = Q K^T and dP = dA V^T for 32 queries x this wave's 32 keys;
        // lane = key, reg i = query qt*32 + krow(i, h2)
        ChFrag<T, D> qa, daa;
        qa.load(&q_lds[(qt * 32 + arow) * RSTR], h2);
        daa.load(&da_lds[(qt * 32 + arow) * RSTR], h2);
        f32x16 S = zero16(), dP = zero16();
        ChFrag<T, D>::mma(S, qa, kb);
        ChFrag<T, D>::mma(dP, daa, vb);
        float bv[16];
        if (brow && bias_vec && (qt + 1) * 32 <= L && (kt + 1) * 32 <= L) {
            // whole tile in range (uniform): two 16-byte loads of bias^T
            load_row8<T>(brow, qt * 32 + 8 * h2, L, true, bv);
            load_row8<T>(brow, qt * 32 + 16 + 8 * h2, L, true, bv + 8);
        } else {
#pragma unroll
            for (int i = 0; i < 16; ++i) bv[i] = 0.0f;
            if (brow && kin) {
                load_row8<T>(brow, qt * 32 + 8 * h2, L, false, bv);
                load_row8<T>(brow, qt * 32 + 16 + 8 * h2, L, false, bv + 8);
            }
        }
        float l2[16], dsv[16];
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int q0 = qt * 32 + 16 * half + 8 * h2;
            const float4 *lp = reinterpret_cast<const float4 *>(&lse2_lds[q0]);
            const float4 *dp = reinterpret_cast<const float4 *>(&dsum_lds[q0]);
            const float4 x0 = lp[0], x1 = lp[1], y0 = dp[0], y1 = dp[1];
            l2[8 * half + 0] = x0.x; l2[8 * half + 1] = x0.y; l2[8 * half + 2] = x0.z; l2[8 * half + 3] = x0.w;
            l2[8 * half + 4] = x1.x; l2[8 * half + 5] = x1.y; l2[8 * half + 6] = x1.z; l2[8 * half + 7] = x1.w;
            dsv[8 * half + 0] = y0.x; dsv[8 * half + 1] = y0.y; dsv[8 * half + 2] = y0.z; dsv[8 * half + 3] = y0.w;
            dsv[8 * half + 4] = y1.x; dsv[8 * half + 5] = y1.y; dsv[8 * half + 6] = y1.z; dsv[8 * half + 7] = y1.w;
        }
        f32x16 P, dS;
        const float keepf = (kfull || kvalid) ? 1.0f : 0.0f;  // masked key: its lane's P is 0
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const float t = __builtin_fmaf(S[i], a.scale, bv[i]);
            const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(t, kLog2e, -l2[i])) * keepf;
            P[i] = p;
            dS[i] = p * (dP[i] - dsv[i]);
        }
        const K32 pb = Tr<T>::pack(P);
        const K32 dsb = Tr<T>::pack(dS);
        // dV^T += dA^T P ;  dK^T += Q^T dS   (A rows: channel sig(n))
        K32 dat, qtf;
        if constexpr (kTr) {
            dat = load_k32_tr(da_lds, RSTR, qt * 32, D, lane);
            qtf = load_k32_tr(q_lds, RSTR, qt * 32, D, lane);
        } else if (arow < D) {
            dat = load_k32<T>(&dat_lds[arow * TSTR + qt * 32], h2);
            qtf = load_k32<T>(&qt_lds[arow * TSTR + qt * 32], h2);
        } else {
            dat = zero_k32<T>();
            qtf = zero_k32<T>();
        }
        Tr<T>::mma_k32(dv_acc, dat, pb);
        Tr<T>::mma_k32(dk_acc, qtf, dsb);
    }

    // ---- dK and dV of this key tile are complete (lane = key, reg = channel)
    if (kin) {
        E *dKp = (E *)a.dk + base + (int64_t)key * a.stok;
        E *dVp = (E *)a.dv + base + (int64_t)key * a.stok;
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int c0 = 16 * half + 8 * h2;
            if (c0 >= D) continue;
            const int o = 8 * half;
            if constexpr (sizeof(E) == 2) {
                uint4 wk, wv;
                uint32_t *pk = reinterpret_cast<uint32_t *>(&wk), *pv = reinterpret_cast<uint32_t *>(&wv);
#pragma unroll
                for (int s = 0; s < 4; ++s) {
                    pk[s] = (uint32_t)f2bf(dk_acc[o + 2 * s] * a.scale) |
                            ((uint32_t)f2bf(dk_acc[o + 2 * s + 1] * a.scale) << 16);
                    pv[s] = (uint32_t)f2bf(dv_acc[o + 2 * s]) | ((uint32_t)f2bf(dv_acc[o + 2 * s + 1]) << 16);
                }
                *reinterpret_cast<uint4 *>(dKp + c0) = wk;
                *reinterpret_cast<uint4 *>(dVp + c0) = wv;
            } else {
                *reinterpret_cast<float4 *>(dKp + c0) = make_float4(
                    dk_acc[o] * a.scale, dk_acc[o + 1] * a.scale, dk_acc[o + 2] * a.scale, dk_acc[o + 3] * a.scale);
                *reinterpret_cast<float4 *>(dKp + c0 + 4) = make_float4(
                    dk_acc[o + 4] * a.scale, dk_acc[o + 5] * a.scale, dk_acc[o + 6] * a.scale, dk_acc[o + 7] * a.scale);
                *reinterpret_cast<float4 *>(dVp + c0) = make_float4(dv_acc[o], dv_acc[o + 1], dv_acc[o + 2], dv_acc[o + 3]);
                *reinterpret_cast<float4 *>(dVp + c0 + 4) =
                    make_float4(dv_acc[o + 4], dv_acc[o + 5], dv_acc[o + 6], dv_acc[o + 7]);
            }
        }
    }
}

// ---------------------------------------------------------------------------
struct QbArgs {
    const void *q, *k, *v, *bias;
    const uint8_t *mask;
    const float *lse;
    const void *da;      // workspace [N][H][L][D]
    const float *dsum;   // workspace [N][H][L]
    void *dq;
    float *part;         // [B][H][chunks][L][L] or null
    int64_t L, rpb, srow, stok, chunks, rows_per_chunk;
    int H;
    float scale;
};

template <typename T, int D, int NKT>
__global__ void __launch_bounds__(NKT * 64) qbias_kernel(QbArgs a) {
    using E = typename Tr<T>::elem;
    using K32 = typename Tr<T>::K32;
    constexpr bool kTr = sizeof(E) == 2;    // bf16: K^T fragments via the transposing LDS read
    constexpr int VEC = Tr<T>::VEC;
    constexpr int CPT = D / VEC;            // 16-byte chunks per token
    constexpr int LP = NKT * 32;
    constexpr int NT = NKT * 64;
    constexpr int KSTR = D + VEC;           // row stride of K, V, Q, dA tiles in LDS (elements)
    constexpr int PSTR = D + 4;             // dQ partial stride in LDS (floats)
    constexpr int NKV = (LP * CPT + NT - 1) / NT;  // 16-byte chunks of K (and of V) per thread
    constexpr int NQC = (32 * CPT + NT - 1) / NT;  // 16-byte chunks of the Q (and dA) tile per thread
    constexpr int NSUM = (32 * (D / 4) + NT - 1) / NT;  // 4-channel groups of dQ summed per thread
    __shared__ __attribute__((aligned(16))) E k_lds[LP * KSTR];
    __shared__ __attribute__((aligned(16))) E v_lds[LP * KSTR];
    __shared__ __attribute__((aligned(16))) E q_lds[32 * KSTR];
    __shared__ __attribute__((aligned(16))) E da_lds[32 * KSTR];
    __shared__ __attribute__((aligned(16))) float lse2_lds[32];
    __shared__ __attribute__((aligned(16))) float dsum_lds[32];
    __shared__ uint32_t kbits_lds[NKT];
    __shared__ __attribute__((aligned(16))) float dqp[NKT * 32 * PSTR];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h2 = lane >> 5, n = lane & 31;
    const int L = (int)a.L;
    const int nqt = (L + 31) / 32;
    // unit -> (b, chunk, qt, head), head fastest
    const int64_t unit = xcd_unit(blockIdx.x, gridDim.x);
    const int hh = (int)(unit % a.H);
    int64_t rest = unit / a.H;
    const int qt = (int)(rest % nqt);
    rest /= nqt;
    const int64_t chunk = rest % a.chunks, b = rest / a.chunks;
    const int64_t r_begin = b * a.rpb + chunk * a.rows_per_chunk;
    int64_t r_end = r_begin + a.rows_per_chunk;
    if (r_end > (b + 1) * a.rpb) r_end = (b + 1) * a.rpb;

    const int kt = wave;
    const int qi = qt * 32 + n;  // this lane's query
    const bool qvalid = qi < L;
    const bool vec_ok = (L % VEC) == 0;

    // bias tile of (this query tile, this key tile): constant over rows
    float bt[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) bt[i] = 0.0f;
    if (a.bias && qvalid) {
        const E *row = (const E *)a.bias + ((b * a.H + hh) * (int64_t)L + qi) * L;
        load_row8<T>(row, kt * 32 + 8 * h2, L, vec_ok, bt);
        load_row8<T>(row, kt * 32 + 16 + 8 * h2, L, vec_ok, bt + 8);
    }
    f32x16 acc = zero16();

    // ---- one row's inputs, staged through registers (loads of row r+1 are in
    // flight while row r is computed)
    uint4 kpf[NKV], vpf[NKV], qpf[NQC], dapf[NQC];
    float lpf = -INFINITY, dspf = 0.0f;
    bool mpf = false;
    auto prefetch = [&](int64_t r) {
        const int64_t base = r * a.srow + (int64_t)hh * D;
        const int64_t rh = r * a.H + hh;
#pragma unroll
        for (int j = 0; j < NKV; ++j) {
            const int idx = tid + j * NT;
            const int t = idx / CPT, c = (idx % CPT) * VEC;
            kpf[j] = make_uint4(0, 0, 0, 0);
            vpf[j] = make_uint4(0, 0, 0, 0);
            if (idx < LP * CPT && t < L) {
                kpf[j] = *reinterpret_cast<const uint4 *>((const E *)a.k + base + (int64_t)t * a.stok + c);
                vpf[j] = *reinterpret_cast<const uint4 *>((const E *)a.v + base + (int64_t)t * a.stok + c);
            }
        }
#pragma unroll
        for (int j = 0; j < NQC; ++j) {
            const int idx = tid + j * NT;
            const int t = qt * 32 + idx / CPT, c = (idx % CPT) * VEC;
            qpf[j] = make_uint4(0, 0, 0, 0);
            dapf[j] = make_uint4(0, 0, 0, 0);
            if (idx < 32 * CPT && t < L) {
                qpf[j] = *reinterpret_cast<const uint4 *>((const E *)a.q + base + (int64_t)t * a.stok + c);
                dapf[j] = *reinterpret_cast<const uint4 *>((const E *)a.da + (rh * L + t) * D + c);
            }
        }
        if (tid < 32) {
            const int t = qt * 32 + tid;
            lpf = t < L ? a.lse[rh * L + t] : -INFINITY;
            dspf = t < L ? a.dsum[rh * L + t] : 0.0f;
        }
        mpf = tid < L && (!a.mask || a.mask[r * a.L + tid] != 0);
    };

    if (r_begin < r_end) prefetch(r_begin);
    for (int64_t r = r_begin; r < r_end; ++r) {
        const int64_t base = r * a.srow + (int64_t)hh * D;
        // ---- registers -> LDS
#pragma unroll
        for (int j = 0; j < NKV; ++j) {
            const int idx = tid + j * NT;
            if (idx < LP * CPT) {
                const int t = idx / CPT, c = (idx % CPT) * VEC;
                *reinterpret_cast<uint4 *>(&k_lds[t * KSTR + c]) = kpf[j];
                *reinterpret_cast<uint4 *>(&v_lds[t * KSTR + c]) = vpf[j];
            }
        }
#pragma unroll
        for (int j = 0; j < NQC; ++j) {
            const int idx = tid + j * NT;
            if (idx < 32 * CPT) {
                const int t = idx / CPT, c = (idx % CPT) * VEC;
                *reinterpret_cast<uint4 *>(&q_lds[t * KSTR + c]) = qpf[j];
                *reinterpret_cast<uint4 *>(&da_lds[t * KSTR + c]) = dapf[j];
            }
        }
        if (tid < 32) {
            lse2_lds[tid] = (lpf == -INFINITY) ? INFINITY : lpf * kLog2e;  // fully masked query: P = 0
            dsum_lds[tid] = dspf;
        }
        {
            const unsigned long long bal = __ballot(mpf);  // NT >= LP: one key per thread
            if (lane == 0) {
                if (2 * wave < NKT) kbits_lds[2 * wave] = (uint32_t)bal;
                if (2 * wave + 1 < NKT) kbits_lds[2 * wave + 1] = (uint32_t)(bal >> 32);
            }
        }
        __syncthreads();
        if (r + 1 < r_end) prefetch(r + 1);

        const uint32_t kbits = __builtin_amdgcn_readfirstlane(kbits_lds[kt]);
        f32x16 dq = zero16();
        if (kbits != 0) {
            ChFrag<T, D> qb, dab, ka, va;
            qb.load(&q_lds[n * KSTR], h2);
            dab.load(&da_lds[n * KSTR], h2);
            ka.load(&k_lds[(kt * 32 + sig(n)) * KSTR], h2);
            va.load(&v_lds[(kt * 32 + sig(n)) * KSTR], h2);
            const float l2 = lse2_lds[n], ds = dsum_lds[n];
            // S^T = K Q^T, dP^T = V dA^T: lane = query, reg i = key kt*32 + krow(i, h2)
            f32x16 S = zero16(), dP = zero16();
            ChFrag<T, D>::mma(S, ka, qb);
            ChFrag<T, D>::mma(dP, va, dab);
            f32x16 dS;
            if (kbits == 0xffffffffu) {
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const float t = __builtin_fmaf(S[i], a.scale, bt[i]);
                    const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(t, kLog2e, -l2));
                    dS[i] = p * (dP[i] - ds);
                    acc[i] += dS[i];
                }
            } else {
                const uint32_t kbl = kbits >> (8 * h2);
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const float t = __builtin_fmaf(S[i], a.scale, bt[i]);
                    float p = __builtin_amdgcn_exp2f(__builtin_fmaf(t, kLog2e, -l2));
                    p = ((kbl >> (16 * (i >> 3) + (i & 7))) & 1u) ? p : 0.0f;
                    dS[i] = p * (dP[i] - ds);
                    acc[i] += dS[i];
                }
            }
            // dQ^T (channels x queries) = K^T dS^T over this wave's keys
            K32 kT;
            if constexpr (kTr) {
                kT = load_k32_tr(k_lds, KSTR, kt * 32, D, lane);
            } else {
                const int c = sig(n);
#pragma unroll
                for (int u = 0; u < 16; ++u) kT.v[u] = c < D ? k_lds[(kt * 32 + krow(u, h2)) * KSTR + c] : 0.0f;
            }
            Tr<T>::mma_k32(dq, kT, Tr<T>::pack(dS));
        }
        // ---- fixed-order sum of the waves' dQ partials through LDS
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int c0 = 16 * half + 8 * h2;
            if (c0 >= D) continue;
            float *dst = &dqp[(wave * 32 + n) * PSTR + c0];
            *reinterpret_cast<float4 *>(dst) = make_float4(dq[8 * half], dq[8 * half + 1], dq[8 * half + 2], dq[8 * half + 3]);
            *reinterpret_cast<float4 *>(dst + 4) =
                make_float4(dq[8 * half + 4], dq[8 * half + 5], dq[8 * half + 6], dq[8 * half + 7]);
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < NSUM; ++j) {  // four consecutive channels per thread and step
            const int idx = tid + j * NT;
            if (idx >= 32 * (D / 4)) break;
            const int q = idx / (D / 4), c = (idx % (D / 4)) * 4;
            float4 s = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll
            for (int w = 0; w < NKT; ++w) {
                const float4 x = *reinterpret_cast<const float4 *>(&dqp[(w * 32 + q) * PSTR + c]);
                s.x += x.x; s.y += x.y; s.z += x.z; s.w += x.w;
            }
            if (qt * 32 + q < L) {
                E *dst = (E *)a.dq + base + (int64_t)(qt * 32 + q) * a.stok + c;
                if constexpr (sizeof(E) == 2) {
                    uint2 w2;
                    w2.x = (uint32_t)f2bf(s.x * a.scale) | ((uint32_t)f2bf(s.y * a.scale) << 16);
                    w2.y = (uint32_t)f2bf(s.z * a.scale) | ((uint32_t)f2bf(s.w * a.scale) << 16);
                    *reinterpret_cast<uint2 *>(dst) = w2;
                } else {
                    *reinterpret_cast<float4 *>(dst) = make_float4(s.x * a.scale, s.y * a.scale, s.z * a.scale, s.w * a.scale);
                }
            }
        }
    }

    // ---- partial dBias tile of this chunk: [qi][kt*32 + krow(i, h2)]
    if (a.part && qvalid) {
        float *pp = a.part + (((b * a.H + hh) * a.chunks + chunk) * (int64_t)L + qi) * L;
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int j0 = kt * 32 + 16 * half + 8 * h2;
            if (j0 + 8 <= L && (L % 4) == 0) {
                *reinterpret_cast<float4 *>(pp + j0) = make_float4(acc[8 * half], acc[8 * half + 1], acc[8 * half + 2], acc[8 * half + 3]);
                *reinterpret_cast<float4 *>(pp + j0 + 4) =
                    make_float4(acc[8 * half + 4], acc[8 * half + 5], acc[8 * half + 6], acc[8 * half + 7]);
            } else {
#pragma unroll
                for (int s = 0; s < 8; ++s)
                    if (j0 + s < L) pp[j0 + s] = acc[8 * half + s];
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
template <typename T, int D, int NKT>
hipError_t launch_passes(const Problem &p, const KvArgs &ka, const QbArgs &qa, const BwdPlan &plan, hipStream_t s,
                         Tracer &tr) {
    hipLaunchKernelGGL((kv_kernel<T, D, NKT>), dim3((unsigned)(p.N * p.H)), dim3(NKT * 64), 0, s, ka);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    tr.mark(s);
    hipLaunchKernelGGL((qbias_kernel<T, D, NKT>), dim3((unsigned)plan.n_wg), dim3(NKT * 64), 0, s, qa);
    e = hipGetLastError();
    if (e == hipSuccess) tr.mark(s);
    return e;
}

template <typename T, int D>
hipError_t launch_passes_d(const Problem &p, const KvArgs &ka, const QbArgs &qa, const BwdPlan &plan, hipStream_t s,
                           Tracer &tr) {
    const int64_t nkt = (p.L + 31) / 32;
    if (nkt <= 1) return launch_passes<T, D, 1>(p, ka, qa, plan, s, tr);
    if (nkt <= 2) return launch_passes<T, D, 2>(p, ka, qa, plan, s, tr);
    if (nkt <= 4) return launch_passes<T, D, 4>(p, ka, qa, plan, s, tr);
    return launch_passes<T, D, 8>(p, ka, qa, plan, s, tr);
}

template <typename T>
hipError_t launch_bwd_t(const Problem &p, const BwdPtrs &x, void *ws, const BwdPlan &plan, hipStream_t s,
                        Tracer &tr) {
    using E = typename Tr<T>::elem;
    char *w = (char *)ws;
    const int64_t planes = x.bias ? (p.N / p.rpb) * p.H : 0;
    hipError_t e;
    tr.mark(s);
    if (x.bias) {
        const int64_t tiles = (p.L + 31) / 32;
        hipLaunchKernelGGL((transpose_kernel<E>), dim3((unsigned)(planes * tiles * tiles)), dim3(256), 0, s,
                           (const E *)x.bias, (E *)(w + plan.off_biast), p.L, tiles);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        tr.mark(s);
    }
    const int64_t rpb = x.bias ? p.rpb : p.N;
    const float scale = 1.0f / sqrtf((float)p.D);
    KvArgs ka;
    ka.q = x.q; ka.k = x.k; ka.v = x.v; ka.g = x.g; ka.out = x.out; ka.dout = x.dout;
    ka.biasT = x.bias ? (const void *)(w + plan.off_biast) : nullptr;
    ka.mask = x.mask; ka.lse = x.lse;
    ka.dk = x.dk; ka.dv = x.dv; ka.dg = x.dg;
    ka.da = w + plan.off_da; ka.dsum = (float *)(w + plan.off_dsum);
    ka.L = p.L; ka.rpb = rpb; ka.srow = p.srow; ka.stok = p.stok; ka.H = p.H; ka.scale = scale;
    QbArgs qa;
    qa.q = x.q; qa.k = x.k; qa.v = x.v; qa.bias = x.bias; qa.mask = x.mask; qa.lse = x.lse;
    qa.da = ka.da; qa.dsum = ka.dsum; qa.dq = x.dq;
    qa.part = x.bias ? (float *)(w + plan.off_part) : nullptr;
    qa.L = p.L; qa.rpb = rpb; qa.srow = p.srow; qa.stok = p.stok;
    qa.chunks = plan.chunks; qa.rows_per_chunk = plan.rows_per_chunk;
    qa.H = p.H; qa.scale = scale;
    switch (p.D) {
        case 8: e = launch_passes_d<T, 8>(p, ka, qa, plan, s, tr); break;
        case 16: e = launch_passes_d<T, 16>(p, ka, qa, plan, s, tr); break;
        default: e = launch_passes_d<T, 32>(p, ka, qa, plan, s, tr); break;
    }
    if (e != hipSuccess || !x.bias) return e;
    const int64_t pe = p.L * p.L;
    int64_t blocks = (planes * pe + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(dbias_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                       (const float *)(w + plan.off_part), x.dbias, planes, plan.chunks, pe);
    e = hipGetLastError();
    if (e == hipSuccess) tr.mark(s);
    return e;
}

}  // namespace

BwdPlan plan_bwd(const Problem &p, bool has_bias) {
    BwdPlan pl;
    const int64_t es = p.dtype == 1 ? 2 : 4;
    const int64_t planes = has_bias ? p.N / p.rpb : (p.N > 0 ? 1 : 0);
    const int64_t rpb = has_bias ? p.rpb : p.N;
    const int64_t nqt = (p.L + 31) / 32;
    const int64_t waves = nqt <= 1 ? 1 : nqt <= 2 ? 2 : nqt <= 4 ? 4 : 8;  // per qbias workgroup
    // qbias workgroups: enough waves to fill the chip (2048 = 8 per CU), with
    // as few row chunks as that allows (each chunk costs one partial dBias plane)
    int64_t target_waves = 2048;
    if (const char *env = getenv("EVO_ATTN_QBIAS_WAVES")) {
        const long v = atol(env);
        if (v > 0) target_waves = v;
    }
    int64_t chunks = 0, g = 1;
    if (planes > 0 && rpb > 0 && nqt > 0) {
        const int64_t per_chunk = planes * p.H * nqt * waves;  // waves per row chunk
        chunks = (target_waves + per_chunk - 1) / per_chunk;
        if (chunks < 1) chunks = 1;
        if (chunks > rpb) chunks = rpb;
        g = (rpb + chunks - 1) / chunks;
        chunks = (rpb + g - 1) / g;
    }
    pl.chunks = chunks;
    pl.rows_per_chunk = g;
    pl.n_wg = planes * p.H * nqt * chunks;
    size_t off = 0;
    pl.off_da = off;
    off = align256(off + (size_t)(p.N * p.L * p.H * p.D * es));
    pl.off_dsum = off;
    off = align256(off + (size_t)(p.N * p.H * p.L) * 4);
    pl.off_biast = off;
    if (has_bias) off = align256(off + (size_t)(planes * p.H * p.L * p.L * es));
    pl.off_part = off;
    if (has_bias) off = align256(off + (size_t)(planes * p.H * chunks * p.L * p.L) * 4);
    pl.total = off;
    return pl;
}

int bwd_kernel_count(bool has_bias) { return has_bias ? 4 : 2; }

hipError_t launch_bwd(const Problem &p, const BwdPtrs &x, void *ws, const BwdPlan &plan, hipStream_t s,
                      Tracer *tr) {
    Tracer none;
    Tracer &t = tr ? *tr : none;
    if (p.dtype == 1) return launch_bwd_t<bf16_t>(p, x, ws, plan, s, t);
    return launch_bwd_t<float>(p, x, ws, plan, s, t);
}

}  // namespace evo
