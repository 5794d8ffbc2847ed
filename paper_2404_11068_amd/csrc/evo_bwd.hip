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
//
// Both passes keep their registers near 120 and their LDS under 80 KB so
// that two 8-wave workgroups share a CU and hide each other's loads and
// barriers.  Global memory is accessed through buffer instructions on
// per-row resources with out-of-range offsets instead of branches (zeros on
// load, dropped stores), so every load is issued unconditionally and in the
// order it is needed.
#include <math.h>
#include <stdlib.h>

#include <atomic>
#include <mutex>

#include "evo_frag.h"
#include "evo_kernels.h"

namespace evo {

namespace {

constexpr float kLog2e = 1.4426950408889634f;

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// 16 bias values of a lane as fp32: reg i <-> element j0 + 16*(i/8) + i%8 of
// the row (the k32 order), from two 8-element groups.  BV: 16-byte aligned
// groups (the row length is a multiple of 16 bytes / element size).
template <typename T, bool BV>
__device__ __forceinline__ void load_bias16(rsrc_t r, uint32_t e0, float *out16) {
    using E = typename Tr<T>::elem;
    constexpr int ES = sizeof(E);
#pragma unroll
    for (int g = 0; g < 2; ++g) {
        const uint32_t e = e0 + 16u * g;
        if constexpr (BV && ES == 2) {
            const u32x4 w = bload16(r, e * 2u);
            const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                out16[8 * g + 2 * s] = __builtin_bit_cast(float, ws[s] << 16);
                out16[8 * g + 2 * s + 1] = __builtin_bit_cast(float, ws[s] & 0xffff0000u);
            }
        } else if constexpr (BV) {
            const f32x4 x0 = __builtin_bit_cast(f32x4, bload16(r, e * 4u));
            const f32x4 x1 = __builtin_bit_cast(f32x4, bload16(r, e * 4u + 16u));
            out16[8 * g + 0] = x0.x; out16[8 * g + 1] = x0.y; out16[8 * g + 2] = x0.z; out16[8 * g + 3] = x0.w;
            out16[8 * g + 4] = x1.x; out16[8 * g + 5] = x1.y; out16[8 * g + 6] = x1.z; out16[8 * g + 7] = x1.w;
        } else if constexpr (ES == 2) {
#pragma unroll
            for (int s = 0; s < 8; ++s) out16[8 * g + s] = bf2f(bload2(r, (e + s) * 2u));
        } else {
#pragma unroll
            for (int s = 0; s < 8; ++s) out16[8 * g + s] = __builtin_bit_cast(float, bload4(r, (e + s) * 4u));
        }
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
    const void *q, *k, *v, *g, *out, *dout;
    const void *bias;   // [planes][H][L][L], read directly (bf16, L % 8 == 0)
    const void *biasT;  // its transpose in the workspace (other cases)
    const uint8_t *mask;
    const float *lse;
    void *dk, *dv, *dg;
    void *da;     // workspace [N][H][L][D]
    float *dsum;  // workspace [N][H][L]
    int64_t L, rpb, srow, stok, n_units;
    int H;
    float scale;
};

// The bias block of (query tile qt, key tile kt) through this wave's own
// LDS tile (bias_block_load / bias_block_transpose_raw in evo_frag.h), as
// fp32 in the logit layout of the kv tile: lane n = key n, register i =
// query krow(i, h).
__device__ __forceinline__ void bias_block_transpose(uint16_t *tile, const u32x4 (&raw)[2], int lane,
                                                     float *out16) {
    const Tr<bf16_t>::K32 f = bias_block_transpose_raw(tile, raw, lane);
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const u32x4 w = __builtin_bit_cast(u32x4, f.v[t]);
        const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2) {
            out16[8 * t + 2 * s2] = __builtin_bit_cast(float, ws[s2] << 16);
            out16[8 * t + 2 * s2 + 1] = __builtin_bit_cast(float, ws[s2] & 0xffff0000u);
        }
    }
}

// KG: key groups per unit.  A unit's NKT key tiles run as KG workgroups of
// NKT / KG waves (each stages all of the unit's queries; the first writes
// dA, dG and Dsum), so that a call with few (row, head) units still fills
// the chip.  Staging then runs in KG passes of the full workgroup's batch.
template <typename T, int D, int NKT, bool BV, int KG>
__global__ void __launch_bounds__(NKT / KG * 64) kv_kernel(KvArgs a) {
    using E = typename Tr<T>::elem;
    using K32 = typename Tr<T>::K32;
    constexpr int ES = sizeof(E);
    constexpr int VEC = Tr<T>::VEC;
    constexpr int CPT = D / VEC;     // 16-byte chunks per token
    constexpr int LP = NKT * 32;
    constexpr int NW = NKT / KG;     // waves (key tiles) per workgroup
    constexpr int NT = NW * 64;
    constexpr int RSTR = D + VEC;    // row-major LDS stride
    constexpr int TSTR = LP + VEC;   // transposed LDS stride
    constexpr int NST = (LP * CPT + NKT * 64 - 1) / (NKT * 64);  // staged 16-byte chunks per thread and pass
    constexpr int NPASS = (LP * CPT + NT * NST - 1) / (NT * NST);  // staging passes
    constexpr int NLB = (LP + NT - 1) / NT;  // lse values per thread
    // output channels per workgroup: head_dim 64 runs as two units per (row,
    // head), both forming S and dP from all 64 channels, each producing 32
    // channels of dK and dV; the first also writes dA, dG and Dsum
    constexpr int DO = D > 32 ? 32 : D;
    constexpr int NHALF = D / DO;
    // bf16: Q^T and dA^T fragments come from the transposing LDS read of the
    // row-major tiles; fp32 keeps explicit transposed copies
    constexpr bool kTr = ES == 2;
    // bf16 with whole 16-byte bias row groups: the bias is read as it lies in
    // memory and transposed per tile in LDS; otherwise from its transpose
    constexpr bool kBD = kTr && BV;
    __shared__ __attribute__((aligned(16))) E q_lds[LP * RSTR];
    __shared__ __attribute__((aligned(16))) E da_lds[LP * RSTR];
    __shared__ __attribute__((aligned(16))) E qt_lds[kTr ? 8 : DO * TSTR];
    __shared__ __attribute__((aligned(16))) E dat_lds[kTr ? 8 : DO * TSTR];
    __shared__ __attribute__((aligned(16))) float lse2_lds[LP];
    __shared__ __attribute__((aligned(16))) float dsum_lds[LP];
    __shared__ __attribute__((aligned(16))) uint16_t bt_lds[kBD ? NW * 32 * 32 : 8];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h2 = lane >> 5, n = lane & 31;
    const int L = (int)a.L;
    const int64_t u = xcd_unit(blockIdx.x, gridDim.x);  // (row, head[, half][, key group]), key group fastest
    if (u >= a.n_units) return;
    const int kg = KG == 1 ? 0 : (int)(u % KG);
    const int64_t unit = u / KG;
    const int ch = NHALF == 1 ? 0 : (int)(unit % NHALF);
    const int c_off = ch * DO;  // first output channel of the unit
    const bool writer = ch == 0 && kg == 0;  // writes the per-token outputs shared by the halves and groups
    const int hh = (int)(unit / NHALF % a.H);
    const int64_t r = unit / NHALF / a.H;
    const int64_t b = r / a.rpb;
    const int64_t rh = r * a.H + hh;
    const bool has_gate = a.g != nullptr, has_mask = a.mask != nullptr,
               has_bias = (kBD ? a.bias : a.biasT) != nullptr;
    const uint32_t stok_b = (uint32_t)(a.stok * ES);
    const uint32_t row_bytes = (uint32_t)(a.L * a.stok * ES);
    const rsrc_t none = make_buf(nullptr, 0u);
    auto tok_buf = [&](const void *X) { return make_buf((const E *)X + r * a.srow + (int64_t)hh * D, row_bytes); };

    // ---- every load of the unit goes out first, in the order of use:
    // this wave's key tile (K, V as B operands, lane = key), its mask, the
    // lse of the staged queries, the staged tokens, the first bias tile
    const int kt = kg * NW + wave;
    const int key = kt * 32 + n;
    const bool kin = key < L;
    const uint32_t key_off = kin ? (uint32_t)key * stok_b : kOOB;
    ChFrag<T, D> kb, vb;
    kb.load(tok_buf(a.k), key_off, h2);
    vb.load(tok_buf(a.v), key_off, h2);
    const uint32_t mbyte = bload1(has_mask ? make_buf(a.mask + r * a.L, (uint32_t)L) : none, (uint32_t)key);
    float lraw[NLB];
#pragma unroll
    for (int j = 0; j < NLB; ++j) {
        const int t = tid + j * NT;
        lraw[j] = __builtin_bit_cast(float, bload4(make_buf(a.lse + rh * L, (uint32_t)L * 4u),
                                                   t < L ? (uint32_t)t * 4u : kOOB));
    }
    u32x4 qv[NST], ov[NST], dov[NST], gv[NST];
    const rsrc_t rq = tok_buf(a.q), ro = tok_buf(a.out), rdo = tok_buf(a.dout), rg = has_gate ? tok_buf(a.g) : none;
    auto load_batch = [&](int pass) {
#pragma unroll
        for (int j = 0; j < NST; ++j) {
            const int idx = tid + (pass * NST + j) * NT;
            const int t = idx / CPT, c = (idx % CPT) * VEC;
            const uint32_t off = (idx < LP * CPT && t < L) ? (uint32_t)t * stok_b + (uint32_t)(c * ES) : kOOB;
            qv[j] = bload16(rq, off);
            ov[j] = bload16(ro, off);
            dov[j] = bload16(rdo, off);
            gv[j] = bload16(rg, off);
        }
    };
    load_batch(0);
    // bias of this lane's key: reg i <-> query qt*32 + krow(i, h2)
    const rsrc_t rbt = has_bias ? make_buf((const E *)(kBD ? a.bias : a.biasT) + (b * a.H + hh) * (int64_t)L * L,
                                           (uint32_t)(L * L * ES))
                                : none;
    const uint32_t bt_e0 = (uint32_t)key * (uint32_t)L + 8u * h2;  // element of query 8*h2 in this key's row
    float bcur[16];
    u32x4 braw[2];  // kBD: raw block of the next query tile
    if constexpr (kBD) bias_block_load(rbt, L, 0, kt, lane, braw);
    else load_bias16<T, BV>(rbt, bt_e0, bcur);

    // ---- stage Q and dA (both layouts); dA, Dsum and dG come from dO, O, G
    {
        const rsrc_t rdg = has_gate ? tok_buf(a.dg) : none;
        const rsrc_t rda = make_buf((E *)a.da + rh * (int64_t)L * D, (uint32_t)(L * D * ES));
        const rsrc_t rds = make_buf(a.dsum + rh * L, (uint32_t)L * 4u);
#pragma unroll
        for (int pass = 0; pass < NPASS; ++pass) {
        if (pass > 0) load_batch(pass);
#pragma unroll
        for (int j = 0; j < NST; ++j) {
            const int idx = tid + (pass * NST + j) * NT;
            const int t = idx / CPT, c = (idx % CPT) * VEC;
            const bool in = idx < LP * CPT;
            const bool valid = in && t < L;
            const E *oe = reinterpret_cast<const E *>(&ov[j]);
            const E *de = reinterpret_cast<const E *>(&dov[j]);
            const E *ge = reinterpret_cast<const E *>(&gv[j]);
            u32x4 dav, dgv;
            E *dae = reinterpret_cast<E *>(&dav);
            E *dge = reinterpret_cast<E *>(&dgv);
            float part = 0.0f;
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                const float o = Tr<T>::to_f(oe[e]), d = Tr<T>::to_f(de[e]);
                part = __builtin_fmaf(d, o, part);
                const float sg = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-Tr<T>::to_f(ge[e]) * kLog2e));
                dae[e] = has_gate ? Tr<T>::from_f(d * sg) : de[e];
                dge[e] = Tr<T>::from_f(d * o * (1.0f - sg));
            }
            // Dsum of the token: sum over its CPT consecutive lanes
#pragma unroll
            for (int off = 1; off < CPT; off <<= 1) part += __shfl_xor(part, off);
            const bool wv = valid && writer;
            const uint32_t toff = wv ? (uint32_t)t * stok_b + (uint32_t)(c * ES) : kOOB;
            bstore16(dgv, rdg, toff);  // dropped without a gate
            bstore16(dav, rda, wv ? (uint32_t)((t * D + c) * ES) : kOOB);
            bstore4(__builtin_bit_cast(uint32_t, part), rds, (wv && c == 0) ? (uint32_t)t * 4u : kOOB);
            if (in) {
                if (c == 0) dsum_lds[t] = valid ? part : 0.0f;
                *reinterpret_cast<u32x4 *>(&q_lds[t * RSTR + c]) = qv[j];
                *reinterpret_cast<u32x4 *>(&da_lds[t * RSTR + c]) = dav;
                if constexpr (!kTr) {
                    const E *qe = reinterpret_cast<const E *>(&qv[j]);
                    const int cq = c - c_off;  // transposed copies: the unit's channels only
                    if (NHALF == 1 || (cq >= 0 && cq < DO)) {
#pragma unroll
                        for (int e = 0; e < VEC; ++e) {
                            qt_lds[(cq + e) * TSTR + t] = qe[e];
                            dat_lds[(cq + e) * TSTR + t] = dae[e];
                        }
                    }
                }
            }
        }
        }
#pragma unroll
        for (int j = 0; j < NLB; ++j) {  // padded or fully masked queries: P = 0
            const int t = tid + j * NT;
            if (t < LP) lse2_lds[t] = (t < L && lraw[j] != -INFINITY) ? lraw[j] * kLog2e : INFINITY;
        }
    }
    const bool kvalid = kin && (!has_mask || mbyte != 0);
    const bool kfull = __ballot(kvalid) == ~0ull;
    // bf16: a masked key's logits get -2^64 from a rank-1 term on its lane's
    // column, so its P is exactly 0 (one small MFMA per tile, issued in every
    // tile: cheaper than a select per logit, and a branch around it costs
    // registers)
    const short mask_neg = kvalid ? (short)0 : kBf16MaskNeg;
    const float c2 = a.scale * kLog2e;
    const int arow = sig(n);  // permuted A-operand row of this lane
    uint16_t *const bt_tile = &bt_lds[kBD ? wave * 1024 : 0];  // (per wave of this workgroup)
    if constexpr (kBD) bias_block_transpose(bt_tile, braw, lane, bcur);
    __syncthreads();

    f32x16 dv_acc = zero16(), dk_acc = zero16();
    const int nqt = (L + 31) / 32;
#pragma unroll
    for (int qt = 0; qt < NKT; ++qt) {
        if (qt >= nqt) break;
        // the next tile's bias goes out first (loads complete in order)
        float bnext[kBD ? 1 : 16];
        if (qt + 1 < NKT) {
            if constexpr (kBD) bias_block_load(rbt, L, qt + 1, kt, lane, braw);
            else load_bias16<T, BV>(rbt, bt_e0 + 32u * (qt + 1), bnext);
        }
        // S = Q K^T (plus the masked-key term) and dP = dA V^T for 32
        // queries x this wave's 32 keys; lane = key, reg i = query
        // qt*32 + krow(i, h2)
        ChFrag<T, D> qa, daa;
        qa.load(&q_lds[(qt * 32 + arow) * RSTR], h2);
        daa.load(&da_lds[(qt * 32 + arow) * RSTR], h2);
        f32x16 S = zero16(), dP = zero16();
        ChFrag<T, D>::mma(S, qa, kb);
        if constexpr (kTr) mma_rank1(S, kBf16One, mask_neg, h2);
        ChFrag<T, D>::mma(dP, daa, vb);
        f32x16 P, dS;
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int q0 = qt * 32 + 16 * half + 8 * h2;
            const f32x4 *lp = reinterpret_cast<const f32x4 *>(&lse2_lds[q0]);
            const f32x4 *dp = reinterpret_cast<const f32x4 *>(&dsum_lds[q0]);
            const f32x4 l0 = lp[0], l1 = lp[1], d0 = dp[0], d1 = dp[1];
            const float l2[8] = {l0.x, l0.y, l0.z, l0.w, l1.x, l1.y, l1.z, l1.w};
            const float ds[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
#pragma unroll
            for (int s8 = 0; s8 < 8; ++s8) {
                const int i = 8 * half + s8;
                // log2 P = c2 * S + log2(e) * bias - lse * log2(e)
                float p = __builtin_amdgcn_exp2f(__builtin_fmaf(S[i], c2, __builtin_fmaf(bcur[i], kLog2e, -l2[s8])));
                // fp32 masked key: its lane's P is exactly 0.  A select, not
                // a product: the lse leaves masked keys out, so exp2 of a
                // masked logit far above it is +inf, and inf * 0 would be NaN
                if constexpr (!kTr) {
                    if (!kfull) p = kvalid ? p : 0.0f;
                }
                P[i] = p;
                dS[i] = p * (dP[i] - ds[s8]);
            }
        }
        const K32 pb = Tr<T>::pack(P);
        const K32 dsb = Tr<T>::pack(dS);
        // dV^T += dA^T P ;  dK^T += Q^T dS   (A rows: channel sig(n))
        K32 dat, qtf;
        if constexpr (kTr) {
            dat = load_k32_tr(da_lds + c_off, RSTR, qt * 32, DO, lane);
            qtf = load_k32_tr(q_lds + c_off, RSTR, qt * 32, DO, lane);
        } else if (arow < DO) {
            dat = load_k32<T>(&dat_lds[arow * TSTR + qt * 32], h2);
            qtf = load_k32<T>(&qt_lds[arow * TSTR + qt * 32], h2);
        } else {
            dat = zero_k32<T>();
            qtf = zero_k32<T>();
        }
        Tr<T>::mma_k32(dv_acc, dat, pb);
        Tr<T>::mma_k32(dk_acc, qtf, dsb);
        if (qt + 1 < NKT) {
            if constexpr (kBD) {
                bias_block_transpose(bt_tile, braw, lane, bcur);
            } else {
#pragma unroll
                for (int i = 0; i < 16; ++i) bcur[i] = bnext[i];
            }
        }
    }

    // ---- dK and dV of this key tile are complete (lane = key, reg = channel)
    const rsrc_t rdk = tok_buf(a.dk), rdv = tok_buf(a.dv);
#pragma unroll
    for (int half = 0; half < 2; ++half) {
        const int c0 = 16 * half + 8 * h2;
        if (16 * half >= DO) continue;
        const uint32_t off = c0 < DO ? key_off + (uint32_t)((c_off + c0) * ES) : kOOB;
        const int o = 8 * half;
        if constexpr (ES == 2) {
            u32x4 wk, wv;
            uint32_t pk[4], pv[4];
#pragma unroll
            for (int s2 = 0; s2 < 4; ++s2) {
                pk[s2] = (uint32_t)f2bf(dk_acc[o + 2 * s2] * a.scale) |
                         ((uint32_t)f2bf(dk_acc[o + 2 * s2 + 1] * a.scale) << 16);
                pv[s2] = (uint32_t)f2bf(dv_acc[o + 2 * s2]) | ((uint32_t)f2bf(dv_acc[o + 2 * s2 + 1]) << 16);
            }
            wk.x = pk[0]; wk.y = pk[1]; wk.z = pk[2]; wk.w = pk[3];
            wv.x = pv[0]; wv.y = pv[1]; wv.z = pv[2]; wv.w = pv[3];
            bstore16(wk, rdk, off);
            bstore16(wv, rdv, off);
        } else {
            const f32x4 k0 = {dk_acc[o] * a.scale, dk_acc[o + 1] * a.scale, dk_acc[o + 2] * a.scale, dk_acc[o + 3] * a.scale};
            const f32x4 k1 = {dk_acc[o + 4] * a.scale, dk_acc[o + 5] * a.scale, dk_acc[o + 6] * a.scale,
                              dk_acc[o + 7] * a.scale};
            const f32x4 v0 = {dv_acc[o], dv_acc[o + 1], dv_acc[o + 2], dv_acc[o + 3]};
            const f32x4 v1 = {dv_acc[o + 4], dv_acc[o + 5], dv_acc[o + 6], dv_acc[o + 7]};
            bstore16(__builtin_bit_cast(u32x4, k0), rdk, off);
            bstore16(__builtin_bit_cast(u32x4, k1), rdk, off + 16u);
            bstore16(__builtin_bit_cast(u32x4, v0), rdv, off);
            bstore16(__builtin_bit_cast(u32x4, v1), rdv, off + 16u);
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
    int64_t L, rpb, srow, stok, chunks, rows_per_chunk, n_units;
    int H;
    float scale;
};

// dQ partials in LDS: row (wave, query) of D floats, 16-byte chunks XOR-
// swizzled so that 16 lanes writing 16 consecutive queries hit 16 distinct
// bank groups
template <int D>
__device__ __forceinline__ int dqp_index(int row, int q, int chunk) {
    constexpr int RPB = 64 / D;  // rows per 256 bytes
    return row * D + 4 * (chunk ^ ((q / RPB) % (D / 4)));
}

template <typename T, int D, int NKT, bool BV>
__global__ void __launch_bounds__(NKT * 64) __attribute__((amdgpu_waves_per_eu(4))) qbias_kernel(QbArgs a) {
    using E = typename Tr<T>::elem;
    using K32 = typename Tr<T>::K32;
    constexpr int ES = sizeof(E);
    constexpr bool kTr = ES == 2;           // bf16: K^T fragments via the transposing LDS read
    constexpr int VEC = Tr<T>::VEC;
    constexpr int CPT = D / VEC;            // 16-byte chunks per token
    constexpr int LP = NKT * 32;
    constexpr int NT = NKT * 64;
    // bf16 rows of 32 channels use the swizzled 64-byte layout (sw32);
    // otherwise rows are padded by one 16-byte chunk
    constexpr bool kSw = kTr && D == 32;
    constexpr int KSTR = kSw ? D : D + VEC;  // row stride of K, V, Q, dA tiles in LDS (elements)
    constexpr int NKV = (LP * CPT + NT - 1) / NT;  // 16-byte chunks of K (and of V) per thread
    constexpr int NQC = (32 * CPT + NT - 1) / NT;  // 16-byte chunks of the Q (and dA) tile per thread
    // output channels per workgroup: head_dim 64 runs as two units per (row
    // chunk, query tile, head), both forming S^T and dP^T from all 64 channels,
    // each producing 32 channels of dQ; the first writes the dBias partial
    constexpr int DO = D > 32 ? 32 : D;
    constexpr int NHALF = D / DO;
    constexpr int NSUM = (32 * (DO / 4) + NT - 1) / NT;  // 4-channel groups of dQ summed per thread
    __shared__ __attribute__((aligned(16))) E k_lds[LP * KSTR];
    __shared__ __attribute__((aligned(16))) E v_lds[LP * KSTR];
    __shared__ __attribute__((aligned(16))) E q_lds[32 * KSTR];
    __shared__ __attribute__((aligned(16))) E da_lds[32 * KSTR];
    __shared__ __attribute__((aligned(16))) float lse2_lds[32];
    __shared__ __attribute__((aligned(16))) float dsum_lds[32];
    __shared__ uint32_t kbits_lds[NKT];
    __shared__ __attribute__((aligned(16))) float dqp[NKT * 32 * DO];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h2 = lane >> 5, n = lane & 31;
    const int L = (int)a.L;
    const int nqt = (L + 31) / 32;
    // unit -> (b, chunk, qt, head[, half]), head fastest
    const int64_t unit = xcd_unit(blockIdx.x, gridDim.x);
    if (unit >= a.n_units) return;
    const int ch = NHALF == 1 ? 0 : (int)(unit % NHALF);
    const int c_off = ch * DO;  // first output channel of the unit
    const int hh = (int)(unit / NHALF % a.H);
    int64_t rest = unit / NHALF / a.H;
    const int qt = (int)(rest % nqt);
    rest /= nqt;
    const int64_t chunk = rest % a.chunks, b = rest / a.chunks;
    const int64_t r_begin = b * a.rpb + chunk * a.rows_per_chunk;
    int64_t r_end = r_begin + a.rows_per_chunk;
    if (r_end > (b + 1) * a.rpb) r_end = (b + 1) * a.rpb;

    const int kt = wave;
    const int qi = qt * 32 + n;  // this lane's query
    const bool qvalid = qi < L;
    const bool has_mask = a.mask != nullptr;
    const uint32_t stok_b = (uint32_t)(a.stok * ES);
    const uint32_t row_bytes = (uint32_t)(a.L * a.stok * ES);
    const rsrc_t none = make_buf(nullptr, 0u);
    const float c2 = a.scale * kLog2e;

    // bias tile of (this query tile, this key tile), constant over rows, as
    // the starting value of the S^T tile: sqrt(d) * bias in fp32, so that
    // c2 * S is the logit in base-2 units; reg i <-> key kt*32 + krow(i, h2)
    f32x16 bacc;
    {
        const rsrc_t rb = a.bias ? make_buf((const E *)a.bias + (b * a.H + hh) * (int64_t)L * L, (uint32_t)(L * L * ES))
                                 : none;
        float btl[16];
        load_bias16<T, BV>(rb, qvalid ? (uint32_t)(qi * L + kt * 32 + 8 * h2) : kOOB / ES, btl);
        float sq_hi, sq_lo;
        sqrt_split(D, sq_hi, sq_lo);
        const float sqd = sq_hi + sq_lo;
#pragma unroll
        for (int i = 0; i < 16; ++i) bacc[i] = sqd * btl[i];
    }
    f32x16 acc = zero16();

    // ---- one row's inputs in registers
    u32x4 kr[NKV], vr[NKV], qr[NQC], dar[NQC];
    float lr = 0.0f, dr = 0.0f;
    uint32_t mr = 0;
    // K and V of the next row are requested during this row's exponentials,
    // the rest (small) before the dQ sum
    auto issue_kv = [&](int64_t r) {
        const rsrc_t rk = make_buf((const E *)a.k + r * a.srow + (int64_t)hh * D, row_bytes);
        const rsrc_t rv = make_buf((const E *)a.v + r * a.srow + (int64_t)hh * D, row_bytes);
#pragma unroll
        for (int j = 0; j < NKV; ++j) {
            const int idx = tid + j * NT;
            const int t = idx / CPT, c = (idx % CPT) * VEC;
            const uint32_t off = (idx < LP * CPT && t < L) ? (uint32_t)t * stok_b + (uint32_t)(c * ES) : kOOB;
            kr[j] = bload16(rk, off);
            vr[j] = bload16(rv, off);
        }
    };
    auto issue_rest = [&](int64_t r) {
        const int64_t rh = r * a.H + hh;
        const rsrc_t rq = make_buf((const E *)a.q + r * a.srow + (int64_t)hh * D, row_bytes);
        const rsrc_t rda = make_buf((const E *)a.da + rh * (int64_t)L * D, (uint32_t)(L * D * ES));
#pragma unroll
        for (int j = 0; j < NQC; ++j) {
            const int idx = tid + j * NT;
            const int t = qt * 32 + idx / CPT, c = (idx % CPT) * VEC;
            const bool ok = idx < 32 * CPT && t < L;
            qr[j] = bload16(rq, ok ? (uint32_t)t * stok_b + (uint32_t)(c * ES) : kOOB);
            dar[j] = bload16(rda, ok ? (uint32_t)((t * D + c) * ES) : kOOB);
        }
        const int tq = qt * 32 + (tid & 31);
        const uint32_t qoff = tq < L ? (uint32_t)tq * 4u : kOOB;
        lr = __builtin_bit_cast(float, bload4(make_buf(a.lse + rh * L, (uint32_t)L * 4u), qoff));
        dr = __builtin_bit_cast(float, bload4(make_buf(a.dsum + rh * L, (uint32_t)L * 4u), qoff));
        mr = bload1(has_mask ? make_buf(a.mask + r * a.L, (uint32_t)L) : none, (uint32_t)tid);
    };

    issue_kv(r_begin);
    issue_rest(r_begin);
    for (int64_t r = r_begin; r < r_end; ++r) {
        const int64_t rn = r + 1 < r_end ? r + 1 : r;  // the last row reloads itself
        // ---- registers -> LDS (the previous row's reads of these tiles ended
        // before its dQ-partial barrier)
#pragma unroll
        for (int j = 0; j < NKV; ++j) {
            const int idx = tid + j * NT;
            if (idx < LP * CPT) {
                const int t = idx / CPT, c = (idx % CPT) * VEC;
                const int o = kSw ? sw32(t, idx % CPT) : t * KSTR + c;
                *reinterpret_cast<u32x4 *>(&k_lds[o]) = kr[j];
                *reinterpret_cast<u32x4 *>(&v_lds[o]) = vr[j];
            }
        }
#pragma unroll
        for (int j = 0; j < NQC; ++j) {
            const int idx = tid + j * NT;
            if (idx < 32 * CPT) {
                const int t = idx / CPT, c = (idx % CPT) * VEC;
                const int o = kSw ? sw32(t, idx % CPT) : t * KSTR + c;
                *reinterpret_cast<u32x4 *>(&q_lds[o]) = qr[j];
                *reinterpret_cast<u32x4 *>(&da_lds[o]) = dar[j];
            }
        }
        if (tid < 32) {
            const bool ok = qt * 32 + tid < L && lr != -INFINITY;
            lse2_lds[tid] = ok ? lr * kLog2e : INFINITY;  // padded or fully masked query: P = 0
            dsum_lds[tid] = dr;
        }
        {
            const bool keep = (!has_mask || mr != 0) && tid < L;
            const unsigned long long bal = __ballot(keep);  // NT >= LP: one key per thread
            if (lane == 0) {
                if (2 * wave < NKT) kbits_lds[2 * wave] = (uint32_t)bal;
                if (2 * wave + 1 < NKT) kbits_lds[2 * wave + 1] = (uint32_t)(bal >> 32);
            }
        }
        __syncthreads();

        const uint32_t kbits = __builtin_amdgcn_readfirstlane(kbits_lds[kt]);
        f32x16 dq = zero16();
        if (kbits != 0) {
            ChFrag<T, D> qb, dab, ka, va;
            if constexpr (kSw) {
                load_sw32(qb, q_lds, n, h2);
                load_sw32(dab, da_lds, n, h2);
                load_sw32(ka, k_lds, kt * 32 + sig(n), h2);
                load_sw32(va, v_lds, kt * 32 + sig(n), h2);
            } else {
                qb.load(&q_lds[n * KSTR], h2);
                dab.load(&da_lds[n * KSTR], h2);
                ka.load(&k_lds[(kt * 32 + sig(n)) * KSTR], h2);
                va.load(&v_lds[(kt * 32 + sig(n)) * KSTR], h2);
            }
            const float l2 = lse2_lds[n], ds = dsum_lds[n];
            // S^T = K Q^T + sqrt(d) bias^T, dP^T = V dA^T: lane = query, reg i = key kt*32 + krow(i, h2)
            f32x16 S = bacc, dP = zero16();
            ChFrag<T, D>::mma(S, ka, qb);
            if constexpr (kTr) {
                if (kbits != 0xffffffffu) {  // masked keys: -2^64 on their rows (row n is key sig(n))
                    const short mv = ((kbits >> sig(n)) & 1u) ? (short)0 : kBf16MaskNeg;
                    // the lane half from an opaque copy, so that the term's
                    // constant operand is formed here: hoisted out of the row
                    // loop it is spilled at this kernel's register cap, and its
                    // reload waits for every load and store in flight
                    const int hq = (int)(opaque_u32((uint32_t)lane) >> 5);
                    mma_rank1(S, mv, kBf16One, hq);
                }
            }
            ChFrag<T, D>::mma(dP, va, dab);
            issue_kv(rn);  // K and V are in LDS: the next row's go out now
            f32x16 dS;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                float p = __builtin_amdgcn_exp2f(__builtin_fmaf(S[i], c2, -l2));
                if (!kTr && kbits != 0xffffffffu) p = __builtin_amdgcn_inverse_ballot_w64(
                                                  ((kbits >> krow(i, 0)) & 1u ? 0x00000000ffffffffull : 0ull) |
                                                  ((kbits >> krow(i, 1)) & 1u ? 0xffffffff00000000ull : 0ull))
                                                  ? p : 0.0f;
                dS[i] = p * (dP[i] - ds);
                acc[i] += dS[i];
            }
            // dQ^T (channels x queries) = K^T dS^T over this wave's keys
            K32 kT;
            if constexpr (kSw) {
                kT = load_k32_tr_sw32(k_lds, kt * 32, lane);
            } else if constexpr (kTr) {
                kT = load_k32_tr(k_lds + c_off, KSTR, kt * 32, DO, lane);
            } else {
                const int c = sig(n);
#pragma unroll
                for (int u = 0; u < 16; ++u)
                    kT.v[u] = c < DO ? k_lds[(kt * 32 + krow(u, h2)) * KSTR + c_off + c] : 0.0f;
            }
            Tr<T>::mma_k32(dq, kT, Tr<T>::pack(dS));
        } else {
            issue_kv(rn);
        }
        // ---- fixed-order sum of the waves' dQ partials through LDS
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int c0 = 16 * half + 8 * h2;
            if (16 * half >= DO) continue;
            if (c0 < DO) {
                const f32x4 x0 = {dq[8 * half], dq[8 * half + 1], dq[8 * half + 2], dq[8 * half + 3]};
                const f32x4 x1 = {dq[8 * half + 4], dq[8 * half + 5], dq[8 * half + 6], dq[8 * half + 7]};
                *reinterpret_cast<f32x4 *>(&dqp[dqp_index<DO>(wave * 32 + n, n, c0 / 4)]) = x0;
                *reinterpret_cast<f32x4 *>(&dqp[dqp_index<DO>(wave * 32 + n, n, c0 / 4 + 1)]) = x1;
            }
        }
        __syncthreads();
        issue_rest(rn);
        const rsrc_t rdq = make_buf((E *)a.dq + r * a.srow + (int64_t)hh * D, row_bytes);
#pragma unroll
        for (int j = 0; j < NSUM; ++j) {  // four consecutive channels per thread and step
            const int idx = tid + j * NT;
            const int q = idx / (DO / 4), cq = idx % (DO / 4);
            const bool ok = idx < 32 * (DO / 4);
            f32x4 sum = {0.0f, 0.0f, 0.0f, 0.0f};
            if (ok) {
                // partials read four at a time and added as fixed trees
                constexpr int G = NKT < 4 ? NKT : 4;
#pragma unroll
                for (int w0 = 0; w0 < NKT; w0 += G) {
                    f32x4 x[G];
#pragma unroll
                    for (int w = 0; w < G; ++w)
                        x[w] = *reinterpret_cast<const f32x4 *>(&dqp[dqp_index<DO>((w0 + w) * 32 + q, q, cq)]);
#pragma unroll
                    for (int st = 1; st < G; st *= 2)
#pragma unroll
                        for (int w = 0; w + st < G; w += 2 * st) x[w] += x[w + st];
                    sum += x[0];
                }
            }
            const uint32_t off = (ok && qt * 32 + q < L)
                                     ? (uint32_t)(qt * 32 + q) * stok_b + (uint32_t)((c_off + 4 * cq) * ES)
                                     : kOOB;
            if constexpr (ES == 2) {
                u32x2 w2;
                w2.x = (uint32_t)f2bf(sum.x * a.scale) | ((uint32_t)f2bf(sum.y * a.scale) << 16);
                w2.y = (uint32_t)f2bf(sum.z * a.scale) | ((uint32_t)f2bf(sum.w * a.scale) << 16);
                __builtin_amdgcn_raw_buffer_store_b64(w2, rdq, off, 0, 0);
            } else {
                bstore16(__builtin_bit_cast(u32x4, sum * a.scale), rdq, off);
            }
        }
    }

    // ---- partial dBias tile of this chunk: [qi][kt*32 + krow(i, h2)]
    if (a.part && ch == 0) {
        const rsrc_t rp = make_buf(a.part + ((b * a.H + hh) * a.chunks + chunk) * (int64_t)L * L, (uint32_t)(L * L * 4));
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int j0 = kt * 32 + 16 * half + 8 * h2;
            if ((L % 8) == 0) {  // 8-key groups wholly in or out of range
                const uint32_t off = (qvalid && j0 < L) ? (uint32_t)(qi * L + j0) * 4u : kOOB;
                const f32x4 x0 = {acc[8 * half], acc[8 * half + 1], acc[8 * half + 2], acc[8 * half + 3]};
                const f32x4 x1 = {acc[8 * half + 4], acc[8 * half + 5], acc[8 * half + 6], acc[8 * half + 7]};
                bstore16(__builtin_bit_cast(u32x4, x0), rp, off);
                bstore16(__builtin_bit_cast(u32x4, x1), rp, off + 16u);
            } else {
#pragma unroll
                for (int s8 = 0; s8 < 8; ++s8) {
                    const float v = acc[8 * half + s8];
                    bstore4(__builtin_bit_cast(uint32_t, v), rp,
                            (qvalid && j0 + s8 < L) ? (uint32_t)(qi * L + j0 + s8) * 4u : kOOB);
                }
            }
        }
    }
}

// The same sums four consecutive elements per thread (planes of a multiple
// of 4 elements): 16-byte loads, four chunks' loads in flight, and still
// chunk order for every element (the same bits as the scalar kernel).
__global__ void __launch_bounds__(256) dbias_reduce4_kernel(const float *__restrict__ part,
                                                         float *__restrict__ dbias, int64_t planes,
                                                         int64_t chunks, int64_t plane_elems) {
    const int64_t quads = plane_elems / 4;
    const int64_t total = planes * quads;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t p = e / quads, x = (e % quads) * 4;
        const float *src = part + p * chunks * plane_elems + x;
        f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
        int64_t c = 0;
        for (; c + 4 <= chunks; c += 4) {
            f32x4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const f32x4 *>(src + (c + u) * plane_elems);
#pragma unroll
            for (int u = 0; u < 4; ++u) acc += v[u];
        }
        for (; c < chunks; ++c) acc += *reinterpret_cast<const f32x4 *>(src + c * plane_elems);
        *reinterpret_cast<f32x4 *>(dbias + p * plane_elems + x) = acc;
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
inline unsigned round8(int64_t n) { return (unsigned)((n + 7) / 8 * 8); }

// bf16 bias rows made of whole 16-byte groups: kv reads the bias as it is
inline bool bias_direct(const Problem &p) { return p.dtype == 1 && p.L % 8 == 0; }

// units per (row, head) of the backward passes: head_dim 64 splits the
// output channels over two workgroups
inline int64_t head_halves(const Problem &p) { return p.D > 32 ? p.D / 32 : 1; }

template <typename T, int D, int NKT, bool BV, int KG>
hipError_t launch_kv(const KvArgs &ka0, hipStream_t s) {
    KvArgs ka = ka0;
    ka.n_units = ka0.n_units * KG;
    hipLaunchKernelGGL((kv_kernel<T, D, NKT, BV, KG>), dim3(round8(ka.n_units)), dim3(NKT / KG * 64), 0, s, ka);
    return hipGetLastError();
}

template <typename T, int D, int NKT, bool BV>
hipError_t launch_passes(const Problem &p, const KvArgs &ka, const QbArgs &qa, hipStream_t s, Tracer &tr) {
    // grids are rounded up to a multiple of 8 for the XCD-aware unit order;
    // surplus workgroups exit at once.  With fewer (row, head) units than
    // two per CU, the dK/dV pass splits each unit's key tiles over two
    // workgroups, over four at 64 units or fewer (at 128 units two were
    // faster than four: each group stages the whole row's Q, dO, O and G)
    hipError_t e;
    if constexpr (NKT >= 4) {
        if (ka.n_units <= 64) e = launch_kv<T, D, NKT, BV, 4>(ka, s);
        else if (ka.n_units < 512) e = launch_kv<T, D, NKT, BV, 2>(ka, s);
        else e = launch_kv<T, D, NKT, BV, 1>(ka, s);
    } else {
        e = launch_kv<T, D, NKT, BV, 1>(ka, s);
    }
    if (e != hipSuccess) return e;
    tr.mark(s);
    hipLaunchKernelGGL((qbias_kernel<T, D, NKT, BV>), dim3(round8(qa.n_units)), dim3(NKT * 64), 0, s, qa);
    e = hipGetLastError();
    if (e == hipSuccess) tr.mark(s);
    return e;
}

template <typename T, int D, int NKT>
hipError_t launch_passes_v(const Problem &p, const KvArgs &ka, const QbArgs &qa, hipStream_t s, Tracer &tr) {
    // BV: bias rows split into whole 16-byte groups
    if (p.L % Tr<T>::VEC == 0) return launch_passes<T, D, NKT, true>(p, ka, qa, s, tr);
    return launch_passes<T, D, NKT, false>(p, ka, qa, s, tr);
}

template <typename T, int D>
hipError_t launch_passes_d(const Problem &p, const KvArgs &ka, const QbArgs &qa, hipStream_t s, Tracer &tr) {
    const int64_t nkt = (p.L + 31) / 32;
    if (nkt <= 1) return launch_passes_v<T, D, 1>(p, ka, qa, s, tr);
    if (nkt <= 2) return launch_passes_v<T, D, 2>(p, ka, qa, s, tr);
    if (nkt <= 4) return launch_passes_v<T, D, 4>(p, ka, qa, s, tr);
    // fp32 at head_dim 64 past 128 keys would need more than the 160 KB of LDS
    // (the ABI rejects it before this point)
    if (nkt <= 8) {
        if constexpr (sizeof(typename Tr<T>::elem) == 4 && D > 32) return hipErrorInvalidValue;
        else return launch_passes_v<T, D, 8>(p, ka, qa, s, tr);
    }
    // 257..512 keys: 16-wave workgroups, bf16 with head_dim <= 32 only (the
    // staged Q and dA of 512 tokens fill the LDS otherwise)
    if constexpr (sizeof(typename Tr<T>::elem) == 2 && D <= 32) return launch_passes_v<T, D, 16>(p, ka, qa, s, tr);
    else return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_bwd_t(const Problem &p, const BwdPtrs &x, void *ws, const BwdPlan &plan, hipStream_t s,
                        Tracer &tr) {
    using E = typename Tr<T>::elem;
    char *w = (char *)ws;
    const int64_t planes = x.bias ? (p.N / p.rpb) * p.H : 0;
    hipError_t e;
    tr.mark(s);
    // the kv pass reads a bf16 bias with whole 16-byte row groups directly
    // (the first traced interval is then empty)
    const bool bias_t = x.bias && !bias_direct(p);
    if (!bias_t && x.bias) tr.mark(s);
    if (bias_t) {
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
    ka.bias = x.bias;
    ka.biasT = bias_t ? (const void *)(w + plan.off_biast) : nullptr;
    ka.mask = x.mask; ka.lse = x.lse;
    ka.dk = x.dk; ka.dv = x.dv; ka.dg = x.dg;
    ka.da = w + plan.off_da; ka.dsum = (float *)(w + plan.off_dsum);
    ka.L = p.L; ka.rpb = rpb; ka.srow = p.srow; ka.stok = p.stok; ka.H = p.H; ka.scale = scale;
    ka.n_units = p.N * p.H * head_halves(p);
    QbArgs qa;
    qa.q = x.q; qa.k = x.k; qa.v = x.v; qa.bias = x.bias; qa.mask = x.mask; qa.lse = x.lse;
    qa.da = ka.da; qa.dsum = ka.dsum; qa.dq = x.dq;
    qa.part = x.bias ? (float *)(w + plan.off_part) : nullptr;
    qa.L = p.L; qa.rpb = rpb; qa.srow = p.srow; qa.stok = p.stok;
    qa.chunks = plan.chunks; qa.rows_per_chunk = plan.rows_per_chunk;
    qa.H = p.H; qa.scale = scale;
    qa.n_units = plan.n_wg;
    switch (p.D) {
        case 8: e = launch_passes_d<T, 8>(p, ka, qa, s, tr); break;
        case 16: e = launch_passes_d<T, 16>(p, ka, qa, s, tr); break;
        case 64: e = launch_passes_d<T, 64>(p, ka, qa, s, tr); break;
        default: e = launch_passes_d<T, 32>(p, ka, qa, s, tr); break;
    }
    if (e != hipSuccess || !x.bias) return e;
    const int64_t pe = p.L * p.L;
    int64_t blocks = (planes * pe + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    if (pe % 4 == 0) {  // (dbias from the ABI and the partial planes are 16-byte aligned)
        int64_t b4 = (planes * pe / 4 + 255) / 256;
        if (b4 > 8192) b4 = 8192;
        hipLaunchKernelGGL(dbias_reduce4_kernel, dim3((unsigned)b4), dim3(256), 0, s,
                           (const float *)(w + plan.off_part), x.dbias, planes, plan.chunks, pe);
    } else {
        hipLaunchKernelGGL(dbias_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                           (const float *)(w + plan.off_part), x.dbias, planes, plan.chunks, pe);
    }
    e = hipGetLastError();
    if (e == hipSuccess) tr.mark(s);
    return e;
}

}  // namespace

BwdPlan plan_bwd(const Problem &p, bool has_bias, size_t cap) {
    if (fused_bwd_supported(p, has_bias)) {
        // single pass: the workspace holds the partial dBias planes only;
        // with a cap, fewer row chunks (fewer planes) until it fits
        BwdPlan pl{};
        pl.fused = true;
        int64_t chunks = 1, g = 1;
        fused_bwd_chunks(p, has_bias, &chunks, &g);
        const int64_t rpb = has_bias ? p.rpb : 1;
        size_t total = has_bias ? fused_bwd_partial_bytes(p, chunks) : 0;
        while (total > cap && chunks > 1) {
            const int64_t fewer = chunks / 2 < chunks - 1 ? chunks / 2 : chunks - 1;
            g = (rpb + fewer - 1) / fewer;
            chunks = (rpb + g - 1) / g;
            total = fused_bwd_partial_bytes(p, chunks);
        }
        pl.chunks = chunks;
        pl.rows_per_chunk = g;
        pl.off_part = 0;
        pl.total = total;
        return pl;
    }
    const int64_t es = p.dtype == 1 ? 2 : 4;
    const int64_t planes = has_bias ? p.N / p.rpb : (p.N > 0 ? 1 : 0);
    const int64_t rpb = has_bias ? p.rpb : p.N;
    const int64_t nqt = (p.L + 31) / 32;
    const int64_t waves = nqt <= 1 ? 1 : nqt <= 2 ? 2 : nqt <= 4 ? 4 : nqt <= 8 ? 8 : 16;  // per qbias workgroup
    // qbias workgroups: enough waves to fill the chip twice over (4096 = two
    // 8-wave workgroups on each of 256 CUs: the kernel's registers and LDS
    // allow two per CU), with as few row chunks as that allows (each chunk
    // costs one partial dBias plane)
    // (read once: the workspace size and the launch must see the same value)
    static const int64_t target_waves = [] {
        const char *env = getenv("EVO_ATTN_QBIAS_WAVES");
        const long v = env ? atol(env) : 0;
        return v > 0 ? (int64_t)v : (int64_t)4096;
    }();
    // With 8-wave or larger workgroups, row chunks of at least four rows:
    // with fewer rows per workgroup the per-workgroup staging of a 256-key row
    // and the reduction of the partial planes cost more than the extra
    // workgroups gain (16 rows over 8 heads: 4 chunks beat 8; one-wave
    // workgroups of 32-key rows gain from every extra chunk instead)
    int64_t chunks = 0;
    if (planes > 0 && rpb > 0 && nqt > 0) {
        const int64_t per_chunk = planes * p.H * nqt * waves * head_halves(p);  // waves per row chunk
        chunks = (target_waves + per_chunk - 1) / per_chunk;
        if (waves >= 8 && chunks > rpb / 4) chunks = rpb / 4;
        if (chunks < 1) chunks = 1;
        if (chunks > rpb) chunks = rpb;
    }
    // workspace layout for a given number of row chunks; with a cap, fewer
    // chunks (fewer partial dBias planes, longer qbias workgroups) until it fits
    auto layout = [&](int64_t want) {
        BwdPlan pl{};
        pl.fused = false;
        int64_t g = 1, c = 0;
        if (want > 0) {
            g = (rpb + want - 1) / want;
            c = (rpb + g - 1) / g;
        }
        pl.chunks = c;
        pl.rows_per_chunk = g;
        pl.n_wg = planes * p.H * nqt * c * head_halves(p);
        size_t off = 0;
        pl.off_da = off;
        off = align256(off + (size_t)(p.N * p.L * p.H * p.D * es));
        pl.off_dsum = off;
        off = align256(off + (size_t)(p.N * p.H * p.L) * 4);
        pl.off_biast = off;
        if (has_bias && !bias_direct(p)) off = align256(off + (size_t)(planes * p.H * p.L * p.L * es));
        pl.off_part = off;
        if (has_bias) off = align256(off + (size_t)(planes * p.H * c * p.L * p.L) * 4);
        pl.total = off;
        return pl;
    };
    BwdPlan pl = layout(chunks);
    while (pl.total > cap && pl.chunks > 1) {
        // halve the chunk count (at least one fewer) and lay out again
        const int64_t fewer = pl.chunks / 2 < pl.chunks - 1 ? pl.chunks / 2 : pl.chunks - 1;
        pl = layout(fewer);
    }
    return pl;
}

int bwd_kernel_count(bool has_bias) { return has_bias ? 4 : 2; }

// ---------------------------------------------------------------------------
// Fixed scratch of evo_attn_bwd_noalloc: one copy per device, resident until
// the process ends.  In host code `noalloc_scratch` names a host-side shadow,
// not device memory; the device address is looked up once per device (with
// that device current) and only that address is ever handed to kernels.
static __device__ __align__(256) unsigned char noalloc_scratch[kNoAllocScratchBytes];
namespace {
constexpr int kMaxDevices = 64;
std::atomic<void *> g_noalloc_ptr[kMaxDevices];  // zero-initialised (static storage)
std::mutex g_noalloc_mu;
}  // namespace

hipError_t noalloc_scratch_ptr(void **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    void *p = g_noalloc_ptr[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(g_noalloc_mu);
        p = g_noalloc_ptr[dev].load(std::memory_order_relaxed);
        if (!p) {
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(noalloc_scratch));
            if (e != hipSuccess) return e;
            if (!p) return hipErrorInvalidSymbol;
            g_noalloc_ptr[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return hipSuccess;
}

hipError_t launch_bwd(const Problem &p, const BwdPtrs &x, void *ws, const BwdPlan &plan, hipStream_t s,
                      Tracer *tr) {
    Tracer none;
    Tracer &t = tr ? *tr : none;
    hipError_t e;
    if (plan.fused) {
        t.mark(s);
        e = launch_bwd_fused(p, x, ws, plan.chunks, plan.rows_per_chunk, s, t);
    } else if (p.dtype == 1) {
        e = launch_bwd_t<bf16_t>(p, x, ws, plan, s, t);
    } else {
        e = launch_bwd_t<float>(p, x, ws, plan, s, t);
    }
    if (e == hipSuccess) t.fill(s);
    return e;
}

}  // namespace evo
