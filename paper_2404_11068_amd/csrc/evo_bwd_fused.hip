// evo_bwd_fused.hip -- single-pass backward of the gated attention with pair
// bias, bf16, head_dim 8 / 16 / 32, gfx950.
//
// Recompute-based backward of o = sigmoid(g) * softmax(s) V with
// s = Q K^T / sqrt(d) + bias + mask (ScaleFold Section 3.3, "Multi Head
// Attention": all of the attention, backward included, in one fused kernel;
// the probabilities are recomputed from the saved log-sum-exp):
//   dA = dO sigmoid(g),  dG = dO o (1 - sigmoid(g)),  Dsum_i = sum_c dO_ic o_ic
//   P  = exp(s - lse),   dP = dA V^T,   dS = P (dP - Dsum)
//   dV = P^T dA,  dK = dS^T Q / sqrt(d),  dQ = dS K / sqrt(d),
//   dBias[plane] = sum over the plane's rows of dS.
//
// Every logit is recomputed once (one exponential per logit in the backward).
// Work unit = (row group, head): a workgroup of one wave per 32-key tile walks
// the rows of its group; per row it stages Q and dA (formed from dO, O and G
// on the way in, with dG and Dsum) in LDS, and each wave, lane = key,
// registers = queries, goes over the query tiles:
//   * S = Q K^T and dP = dA V^T on the matrix unit, P and dS in registers;
//   * dV += dA^T P and dK += Q^T dS stay in registers until the row ends;
//   * dQ of the query tile = sum over the key tiles of dS K: each wave turns
//     its dS tile around through a 2 KB LDS tile of its own (transposing read),
//     forms its 32 x d share on the matrix unit, and the shares of the waves
//     are added in a fixed order through a double-buffered LDS area (one
//     barrier per query tile);
//   * dBias: dS accumulates in registers over the rows of the group (the
//     wave's 32 keys x all queries of the plane), and the group writes one
//     partial plane (or, with one group per plane, dBias itself).
// The partial planes are summed in group order by dbias_tiles_reduce_kernel.
// Every sum has a fixed order, so results are bitwise repeatable.
//
// Rows are grouped so that the heads of one group run next to each other on
// one XCD (they share the cache lines of the [H, d] token blocks), and there
// are about 2048 waves in all (one 8-wave workgroup per CU when the bias
// accumulators take half of the register file).
#include <math.h>

#include "evo_frag.h"
#include "evo_kernels.h"

namespace evo {

namespace {

constexpr float kLog2e = 1.4426950408889634f;

struct FusedArgs {
    const void *q, *k, *v, *g, *out, *dout, *bias;
    const uint8_t *mask;
    const float *lse;
    void *dq, *dk, *dv, *dg;
    float *dbias;  // [planes][H][L][L] fp32, written directly when chunks == 1
    float *part;   // [planes][chunks][H][tiles][64 lanes][16] fp32 when chunks > 1
    int64_t L, rpb, srow, stok, chunks, rows_per_chunk, n_units;
    int H;
    float scale;
};

// dQ partials in LDS: row (wave, query) of D floats, 16-byte chunks XOR-
// swizzled so that 16 lanes writing 16 consecutive queries hit 16 distinct
// bank groups
template <int D>
__device__ __forceinline__ int dqs_index(int row, int q, int chunk) {
    constexpr int RPB = 64 / D;  // rows per 256 bytes
    return row * D + 4 * (chunk ^ ((q / RPB) % (D / 4)));
}

// dS (lane = key n, register i = query krow(i, h), packed bf16) into the
// wave's swizzled 32 x 32 tile X[key][column], query q in column sig(q):
// registers 8t + 4u + e (query 16t + 8h + 4u + e) go to column
// 16t + 8u + 4h + e, i.e. chunk 2t + u, elements 4h .. 4h+3.  Read back with
// load_k32_tr_sw32 the tile gives lane n the query sig(sig(n)) = n with the
// keys in its k-slots: the B operand of dQ^T = K^T dS^T.
__device__ __forceinline__ Tr<bf16_t>::K32 ds_transpose(uint16_t *tile, const Tr<bf16_t>::K32 &ds, int n, int h) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const u32x4 w = __builtin_bit_cast(u32x4, ds.v[t]);
        const u32x2 lo = {w.x, w.y}, hi = {w.z, w.w};
        *reinterpret_cast<u32x2 *>(&tile[sw32(n, 2 * t) + 4 * h]) = lo;
        *reinterpret_cast<u32x2 *>(&tile[sw32(n, 2 * t + 1) + 4 * h]) = hi;
    }
    return load_k32_tr_sw32(tile, 0, (h << 5) | n);
}

// dBias accumulators of the query tiles qt >= NQR live in LDS (a wave's own
// region, [tile][4-float group][lane][4], so that a lane's 16-byte accesses are
// bank-conflict free); the first NQR tiles in registers.
template <int NKT, int NQR>
constexpr int kLdsBiasTiles = NKT > NQR ? NKT - NQR : 0;

template <int D, int NKT, bool HB, bool BV, int NQR>
__global__ void __launch_bounds__(NKT * 64) bwd_fused_kernel(FusedArgs a) {
    using E = uint16_t;
    using K32 = Tr<bf16_t>::K32;
    constexpr int ES = 2;
    constexpr int VEC = 8;             // elements per 16 bytes
    constexpr int CPT = D / VEC;       // 16-byte chunks per token
    constexpr int LP = NKT * 32;
    constexpr int NT = NKT * 64;
    constexpr int RSTR = D + VEC;      // row stride of the Q, dA and K tiles in LDS (elements)
    constexpr int NST = (LP * CPT + NT - 1) / NT;           // staged 16-byte chunks per thread
    constexpr int NSUM = (32 * (D / 4) + NT - 1) / NT;      // 4-channel groups of dQ summed per thread
    // head_dim 8: S and dP on the k=16 instruction, whose k-slots 8..15 carry
    // the masked-key term (1 in each Q row's slot 8, the key's -2^64 or 0 in
    // the K operand's) and -Dsum (each dA row's slots 8..10 hold -Dsum as
    // three bf16 terms, the V operand's are 1): S comes with the mask and dP
    // as dP - Dsum, so dS is one multiply per logit
    constexpr bool kPad8 = D == 8;
    using QKF = typename QKFragSel<bf16_t, D>::type;
    static_assert(!kPad8 || CPT == 1, "one 16-byte chunk per token");
    __shared__ __attribute__((aligned(16))) E q_lds[LP * RSTR];
    __shared__ __attribute__((aligned(16))) E da_lds[LP * RSTR];
    __shared__ __attribute__((aligned(16))) E k_lds[LP * RSTR];
    __shared__ __attribute__((aligned(16))) float lse2_lds[LP];
    __shared__ __attribute__((aligned(16))) float dsum_lds[LP];
    __shared__ __attribute__((aligned(16))) uint16_t tp_lds[NKT * 32 * 32];  // per-wave transpose tiles
    __shared__ __attribute__((aligned(16))) float dqp[2][NKT * 32 * D];      // dQ partials, double-buffered
    constexpr int NLB = HB ? kLdsBiasTiles<NKT, NQR> : 0;
    __shared__ __attribute__((aligned(16))) float db_lds[NLB > 0 ? NKT * NLB * 1024 : 4];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int h2 = lane >> 5, n = lane & 31;
    const int L = (int)a.L;
    const int nqt = (L + 31) / 32;
    // unit -> (plane b, row chunk, head), head fastest: the heads of one
    // chunk land on one XCD (xcd_unit) and share the token cache lines
    const int64_t unit = xcd_unit(blockIdx.x, gridDim.x);
    if (unit >= a.n_units) return;
    const int hh = (int)(unit % a.H);
    const int64_t bc = unit / a.H;
    const int64_t chunk = bc % a.chunks, b = bc / a.chunks;
    const int64_t r_begin = b * a.rpb + chunk * a.rows_per_chunk;
    int64_t r_end = r_begin + a.rows_per_chunk;
    if (r_end > (b + 1) * a.rpb) r_end = (b + 1) * a.rpb;

    const bool has_gate = a.g != nullptr, has_mask = a.mask != nullptr;
    const uint32_t stok_b = (uint32_t)(a.stok * ES);
    const uint32_t row_bytes = (uint32_t)(a.L * a.stok * ES);
    const rsrc_t none = make_buf(nullptr, 0u);
    const float c2 = a.scale * kLog2e;
    const int kt = wave;
    const int key = kt * 32 + n;
    const bool kin = key < L;
    const uint32_t key_off = kin ? (uint32_t)key * stok_b : kOOB;
    const rsrc_t rb = HB ? make_buf((const E *)a.bias + (b * a.H + hh) * (int64_t)L * L, (uint32_t)(L * L * ES))
                         : none;
    uint16_t *const tp = &tp_lds[wave * 1024];
    // sqrt(d) on an identity, for the bias product (two bf16 terms where
    // sqrt(d) has no exact bf16 value; their sum matches it to ~3e-7)
    float sq_hi, sq_lo;
    sqrt_split(D, sq_hi, sq_lo);
    const bool two_term = sq_lo != 0.0f;
    K32 eye_hi{}, eye_lo{};
    if constexpr (HB) {
        eye_hi = eye_k32(sq_hi, lane);
        if (two_term) eye_lo = eye_k32(sq_lo, lane);
    }

    // dS of this wave's keys summed over the rows of the chunk, per query
    // tile: tiles below NQR in registers, the rest in the wave's LDS region
    constexpr int NRB = HB ? (NKT < NQR ? NKT : NQR) : 1;
    f32x16 dB[NRB > 0 ? NRB : 1];
    float *const dbl = &db_lds[NLB > 0 ? wave * NLB * 1024 : 0];
    if constexpr (HB) {
#pragma unroll
        for (int t = 0; t < NRB; ++t) dB[t] = zero16();
#pragma unroll
        for (int t = 0; t < NLB; ++t)
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4)
                *reinterpret_cast<f32x4 *>(&dbl[(t * 4 + g4) * 256 + lane * 4]) = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    }

    for (int64_t r = r_begin; r < r_end; ++r) {
        auto tok_buf = [&](const void *X) {
            return make_buf((const E *)X + r * a.srow + (int64_t)hh * D, row_bytes);
        };
        // per-row opaque copies of the lane's bias-row offset (query sig(n) of
        // tile 0, this wave's keys) and lane index: each query tile's bias
        // and dQ addresses are formed from them inside the tile's step
        const uint32_t boff = opaque_u32((uint32_t)((sig(n) * L + kt * 32 + 8 * h2) * ES));
        const uint32_t lane_r = opaque_u32((uint32_t)lane);
        // ---- every load of the row goes out first, in the order of use
        QKF kb, vb;
        if constexpr (kPad8) {
            kb.load(tok_buf(a.k), key_off, h2, (short)0);  // slot 8: the mask word, set below
            vb.load(tok_buf(a.v), key_off, h2, 0x3F803F80u, 0x00003F80u);  // slots 8..10: 1
        } else {
            kb.load(tok_buf(a.k), key_off, h2);
            vb.load(tok_buf(a.v), key_off, h2);
        }
        const uint32_t mbyte = bload1(has_mask ? make_buf(a.mask + r * a.L, (uint32_t)L) : none, (uint32_t)key);
        const float lraw = __builtin_bit_cast(
            float, bload4(make_buf(a.lse + (r * a.H + hh) * L, (uint32_t)L * 4u), tid < L ? (uint32_t)tid * 4u : kOOB));
        u32x4 qv[NST], ov[NST], dov[NST], gv[NST];
        {
            const rsrc_t rq = tok_buf(a.q), ro = tok_buf(a.out), rdo = tok_buf(a.dout),
                         rg = has_gate ? tok_buf(a.g) : none;
#pragma unroll
            for (int j = 0; j < NST; ++j) {
                const int idx = tid + j * NT;
                const int t = idx / CPT, c = (idx % CPT) * VEC;
                const uint32_t off = (idx < LP * CPT && t < L) ? (uint32_t)t * stok_b + (uint32_t)(c * ES) : kOOB;
                qv[j] = bload16(rq, off);
                ov[j] = bload16(ro, off);
                dov[j] = bload16(rdo, off);
                gv[j] = bload16(rg, off);
            }
        }
        // first query tile's bias rows
        K32 bnext;
        if constexpr (HB) {
            if constexpr (BV) bnext = bias_rows_k32_at(rb, boff);
            else bnext = bias_rows_k32<BV>(rb, L, 0, kt, lane);
        }

        // ---- staging: Q and dA into LDS; dA, Dsum and dG from dO, O and G
        {
            const rsrc_t rdg = has_gate ? tok_buf(a.dg) : none;
#pragma unroll
            for (int j = 0; j < NST; ++j) {
                const int idx = tid + j * NT;
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
                    const float o = bf2f(oe[e]), d = bf2f(de[e]);
                    part = __builtin_fmaf(d, o, part);
                    const float sg = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-bf2f(ge[e]) * kLog2e));
                    dae[e] = has_gate ? f2bf(d * sg) : de[e];
                    dge[e] = f2bf(d * o * (1.0f - sg));
                }
                // Dsum of the token: sum over its CPT consecutive lanes
#pragma unroll
                for (int off = 1; off < CPT; off <<= 1) part += __shfl_xor(part, off);
                bstore16(dgv, rdg, valid ? (uint32_t)t * stok_b + (uint32_t)(c * ES) : kOOB);  // dropped without a gate
                if (in) {
                    if (c == 0) dsum_lds[t] = valid ? part : 0.0f;
                    *reinterpret_cast<u32x4 *>(&q_lds[t * RSTR + c]) = qv[j];
                    *reinterpret_cast<u32x4 *>(&da_lds[t * RSTR + c]) = dav;
                    if constexpr (kPad8) {
                        // slots 8..15: Q (1, 0, ...), dA (-Dsum as hi + mid + lo, 0, ...)
                        const float dsv = valid ? part : 0.0f;
                        const uint16_t dh = f2bf(dsv);
                        const float r1 = dsv - bf2f(dh);
                        const uint16_t dm = f2bf(r1);
                        const uint16_t dl = f2bf(r1 - bf2f(dm));
                        const u32x4 qp = {(uint32_t)(uint16_t)kBf16One, 0u, 0u, 0u};
                        const u32x4 dp = {((uint32_t)dh | ((uint32_t)dm << 16)) ^ 0x80008000u, (uint32_t)dl ^ 0x8000u, 0u, 0u};
                        *reinterpret_cast<u32x4 *>(&q_lds[t * RSTR + 8]) = qp;
                        *reinterpret_cast<u32x4 *>(&da_lds[t * RSTR + 8]) = dp;
                    }
                }
            }
            if (tid < LP)  // padded or fully masked queries: P = 0
                lse2_lds[tid] = (tid < L && lraw != -INFINITY) ? lraw * kLog2e : INFINITY;
            // this wave's key rows of K, for the K^T operand of the dQ product
            E *krow_p = &k_lds[key * RSTR];
            if constexpr (kPad8) {
                *reinterpret_cast<bf16x8 *>(krow_p + 8 * h2) = kb.v;  // slots 8..15 are never read
            } else {
#pragma unroll
                for (int kk = 0; kk < D / 16; ++kk)
                    *reinterpret_cast<bf16x8 *>(krow_p + 16 * kk + 8 * h2) = kb.v[kk];
            }
        }
        const bool kvalid = kin && (!has_mask || mbyte != 0);
        const uint64_t kbal = __ballot(kvalid);
        const bool kfull = kbal == ~0ull, kany = kbal != 0ull;
        const short mask_neg = kvalid ? (short)0 : kBf16MaskNeg;  // rank-1 term on this lane's key column
        if constexpr (kPad8) kb.set_slot8(h2, mask_neg);
        // the bias term of query tile 0 (sqrt(d) * bias through the matrix
        // unit), formed while the staging barrier is waited for; each later
        // tile's is formed before the previous tile's dQ barrier
        f32x16 T = zero16();
        if constexpr (HB) {
            Tr<bf16_t>::mma_k32(T, bnext, eye_hi);
            if (two_term) Tr<bf16_t>::mma_k32(T, bnext, eye_lo);
        }
        __syncthreads();

        f32x16 dv_acc = zero16(), dk_acc = zero16();
        const rsrc_t rdq = tok_buf(a.dq);
#pragma unroll
        for (int qt = 0; qt < NKT; ++qt) {
            if (qt >= nqt) break;
            float *const dq_part = dqp[qt & 1];
            // the next tile's bias rows go out first (loads complete in order)
            if constexpr (HB) {
                if (qt + 1 < NKT) {
                    if constexpr (BV) bnext = bias_rows_k32_at(rb, boff + (uint32_t)((qt + 1) * 32 * L * ES));
                    else bnext = bias_rows_k32<BV>(rb, L, qt + 1, kt, lane);
                }
            }
            f32x16 dq = zero16();
            if (kany) {
                // raw logits S = sqrt(d) * bias + Q K^T (the bias term T was
                // formed on the matrix unit before this tile, sqrt(d) as one
                // or two bf16 terms; masked keys get -2^64 from a rank-1
                // term, at head_dim 8 from the product's k-slot 8) and
                // dP = dA V^T (at head_dim 8 already less Dsum), for 32
                // queries x this wave's 32 keys; lane = key, reg i = query
                // qt*32 + krow(i, h2)
                f32x16 S = T, dP = zero16();
                {
                    QKF qa, daa;
                    qa.load(&q_lds[(qt * 32 + sig(n)) * RSTR], h2);
                    daa.load(&da_lds[(qt * 32 + sig(n)) * RSTR], h2);
                    QKF::mma(S, qa, kb);
                    if (!kPad8 && !kfull) mma_rank1(S, kBf16One, mask_neg, h2);
                    QKF::mma(dP, daa, vb);
                }
                f32x16 P, dS;
#pragma unroll
                for (int half = 0; half < 2; ++half) {
                    const int q0 = qt * 32 + 16 * half + 8 * h2;
                    const f32x4 *lp = reinterpret_cast<const f32x4 *>(&lse2_lds[q0]);
                    const f32x4 l0 = lp[0], l1 = lp[1];
                    const float l2[8] = {l0.x, l0.y, l0.z, l0.w, l1.x, l1.y, l1.z, l1.w};
                    float ds[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};  // in dP already at head_dim 8
                    if constexpr (!kPad8) {
                        const f32x4 *dp = reinterpret_cast<const f32x4 *>(&dsum_lds[q0]);
                        const f32x4 d0 = dp[0], d1 = dp[1];
                        ds[0] = d0.x; ds[1] = d0.y; ds[2] = d0.z; ds[3] = d0.w;
                        ds[4] = d1.x; ds[5] = d1.y; ds[6] = d1.z; ds[7] = d1.w;
                    }
#pragma unroll
                    for (int s8 = 0; s8 < 8; ++s8) {
                        const int i = 8 * half + s8;
                        // log2 P = c2 * S_raw - lse * log2(e); a masked key's
                        // S_raw is below -2^63, so its P is exactly 0
                        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(S[i], c2, -l2[s8]));
                        P[i] = p;
                        dS[i] = kPad8 ? p * dP[i] : p * (dP[i] - ds[s8]);
                    }
                }
                if constexpr (HB) {
                    if (qt < NRB) {
#pragma unroll
                        for (int i = 0; i < 16; ++i) dB[qt < NRB ? qt : 0][i] += dS[i];
                    } else {
                        const int t = qt - NRB;
#pragma unroll
                        for (int g4 = 0; g4 < 4; ++g4) {
                            f32x4 *pa = reinterpret_cast<f32x4 *>(&dbl[(t * 4 + g4) * 256 + lane * 4]);
                            const f32x4 o = *pa;
                            *pa = f32x4{o.x + dS[4 * g4], o.y + dS[4 * g4 + 1], o.z + dS[4 * g4 + 2], o.w + dS[4 * g4 + 3]};
                        }
                    }
                }
                const K32 pb = Tr<bf16_t>::pack(P);
                const K32 dsb = Tr<bf16_t>::pack(dS);
                // dV^T += dA^T P ;  dK^T += Q^T dS   (A rows: channel sig(n))
                {
                    // (operand rows of channels >= D only reach output
                    // rows that are never stored: no zeroing needed)
                    const K32 dat = load_k32_tr(da_lds, RSTR, qt * 32, D, lane, false, false);
                    Tr<bf16_t>::mma_k32(dv_acc, dat, pb);
                    const K32 qtf = load_k32_tr(q_lds, RSTR, qt * 32, D, lane, false, false);
                    Tr<bf16_t>::mma_k32(dk_acc, qtf, dsb);
                }
                // dQ^T share of this key tile = K^T dS^T (lane = query n, reg
                // i = channel krow(i, h2))
                const K32 dsT = ds_transpose(tp, dsb, n, h2);
                const K32 kT = load_k32_tr(k_lds, RSTR, kt * 32, D, lane, false, false);
                Tr<bf16_t>::mma_k32(dq, kT, dsT);
            }
            // ---- this wave's dQ share into LDS; fixed-order sum over the waves
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int c0 = 16 * half + 8 * h2;
                if (16 * half >= D) continue;
                if (c0 < D) {
                    const f32x4 x0 = {dq[8 * half], dq[8 * half + 1], dq[8 * half + 2], dq[8 * half + 3]};
                    const f32x4 x1 = {dq[8 * half + 4], dq[8 * half + 5], dq[8 * half + 6], dq[8 * half + 7]};
                    *reinterpret_cast<f32x4 *>(&dq_part[dqs_index<D>(wave * 32 + n, n, c0 / 4)]) = x0;
                    *reinterpret_cast<f32x4 *>(&dq_part[dqs_index<D>(wave * 32 + n, n, c0 / 4 + 1)]) = x1;
                }
            }
            // the next tile's bias term, on the matrix unit while this wave
            // waits at the dQ barrier
            if constexpr (HB) {
                if (qt + 1 < NKT) {
                    T = zero16();
                    Tr<bf16_t>::mma_k32(T, bnext, eye_hi);
                    if (two_term) Tr<bf16_t>::mma_k32(T, bnext, eye_lo);
                }
            }
            __syncthreads();
            // the sum of tile qt is taken by the waves from wave qt % NKT on,
            // as many as its 8·D four-channel groups need: a wave-uniform
            // test, so the other waves skip the index arithmetic and the
            // reads.  Every wave still issues its store (off the end of the
            // buffer where it has nothing to write), so that the count of
            // loads and stores in flight is the same on both sides of the test
            const uint32_t wr = (uint32_t)(wave + NKT - qt % NKT) % NKT;
#pragma unroll
            for (int j = 0; j < NSUM; ++j) {  // four consecutive channels per thread and step
                const uint32_t base = wr * 64u + (uint32_t)(j * NT);  // wave-uniform
                u32x2 w2 = {0u, 0u};
                uint32_t off = kOOB;
                if (base < (uint32_t)(32 * (D / 4))) {
                    const uint32_t idx = base + lane_r;
                    const int q = (int)(idx / (D / 4)), cq = (int)(idx % (D / 4));
                    f32x4 sum = {0.0f, 0.0f, 0.0f, 0.0f};
                    // partials read four at a time and added as fixed trees
                    constexpr int G = NKT < 4 ? NKT : 4;
#pragma unroll
                    for (int w0 = 0; w0 < NKT; w0 += G) {
                        f32x4 x[G];
#pragma unroll
                        for (int w = 0; w < G; ++w)
                            x[w] = *reinterpret_cast<const f32x4 *>(&dq_part[dqs_index<D>((w0 + w) * 32 + q, q, cq)]);
#pragma unroll
                        for (int st = 1; st < G; st *= 2)
#pragma unroll
                            for (int w = 0; w + st < G; w += 2 * st) x[w] += x[w + st];
                        sum += x[0];
                    }
                    if (qt * 32 + q < L) off = (uint32_t)(qt * 32 + q) * stok_b + (uint32_t)(4 * cq * ES);
                    w2.x = (uint32_t)f2bf(sum.x * a.scale) | ((uint32_t)f2bf(sum.y * a.scale) << 16);
                    w2.y = (uint32_t)f2bf(sum.z * a.scale) | ((uint32_t)f2bf(sum.w * a.scale) << 16);
                }
                __builtin_amdgcn_raw_buffer_store_b64(w2, rdq, off, 0, 0);
            }
        }

        // ---- dK and dV of this key tile are complete (lane = key, reg = channel)
        const rsrc_t rdk = tok_buf(a.dk), rdv = tok_buf(a.dv);
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int c0 = 16 * half + 8 * h2;
            if (16 * half >= D) continue;
            const uint32_t off = c0 < D ? key_off + (uint32_t)(c0 * ES) : kOOB;
            const int o = 8 * half;
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
        }
    }

    // ---- the chunk's dBias: one partial plane in tile order [tile][lane][16]
    // (reduced across chunks afterwards), or with one chunk per plane dBias
    // itself, [q][k]
    // (a wave whose key tile lies wholly past L has no tiles of its own)
    if (HB && kt < nqt) {
        const int64_t tiles = (int64_t)nqt * nqt;
        const rsrc_t rp = a.part ? make_buf(a.part + ((b * a.chunks + chunk) * a.H + hh) * tiles * 1024,
                                            (uint32_t)(tiles * 1024 * 4))
                                 : none;
        const rsrc_t rd = a.part ? none : make_buf(a.dbias + (b * a.H + hh) * (int64_t)L * L, (uint32_t)L * L * 4u);
#pragma unroll
        for (int qt = 0; qt < NKT; ++qt) {
            if (qt >= nqt) break;
            f32x16 dbt;
            if (qt < NRB) {
                dbt = dB[qt < NRB ? qt : 0];
            } else {
                const int t = qt - NRB;
#pragma unroll
                for (int g4 = 0; g4 < 4; ++g4) {
                    const f32x4 o = *reinterpret_cast<const f32x4 *>(&dbl[(t * 4 + g4) * 256 + lane * 4]);
                    dbt[4 * g4] = o.x; dbt[4 * g4 + 1] = o.y; dbt[4 * g4 + 2] = o.z; dbt[4 * g4 + 3] = o.w;
                }
            }
            if (a.part) {
                const uint32_t base = (uint32_t)(((qt * nqt + kt) * 1024 + lane * 16) * 4);
#pragma unroll
                for (int g4 = 0; g4 < 4; ++g4) {
                    const f32x4 x = {dbt[4 * g4], dbt[4 * g4 + 1], dbt[4 * g4 + 2], dbt[4 * g4 + 3]};
                    bstore16(__builtin_bit_cast(u32x4, x), rp, base + 16u * g4);
                }
            } else {
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int qi = qt * 32 + krow(i, h2);
                    // through a scalar: a bit-cast of a vector component reads
                    // component 0 with this compiler
                    const float v = dbt[i];
                    bstore4(__builtin_bit_cast(uint32_t, v), rd, (qi < L && kin) ? (uint32_t)(qi * L + key) * 4u : kOOB);
                }
            }
        }
    }
}

// dbias[p][q][k] = sum over chunks c of the tile-ordered partial planes, in
// chunk order.  One workgroup per (plane-head, tile): four waves each sum a
// quarter of the chunks (fixed order), then wave 0 adds the four in order.
__global__ void __launch_bounds__(256) dbias_tiles_reduce_kernel(const float *__restrict__ part,
                                                                 float *__restrict__ dbias, int64_t planes,
                                                                 int H, int64_t chunks, int L) {
    __shared__ __attribute__((aligned(16))) float red[3][64 * 16];
    const int nqt = (L + 31) / 32;
    const int64_t tiles = (int64_t)nqt * nqt;
    const int64_t blk = blockIdx.x;
    const int64_t tile = blk % tiles, ph = blk / tiles;  // ph = plane * H + head
    const int64_t b = ph / H, hh = ph % H;
    const int qt = (int)(tile / nqt), kt = (int)(tile % nqt);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int64_t per = (chunks + 3) / 4;
    const int64_t c0 = wave * per, c1 = c0 + per < chunks ? c0 + per : chunks;
    f32x4 acc[4];
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) acc[g4] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    // element (b, c, hh, tile, lane, i) of the partials
    const int64_t stride_c = (int64_t)H * tiles * 1024;
    const float *src = part + (b * chunks * H + hh) * tiles * 1024 + tile * 1024 + lane * 16;
    int64_t c = c0;
    for (; c + 2 <= c1; c += 2) {
        f32x4 x[2][4];
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4)
                x[u][g4] = *reinterpret_cast<const f32x4 *>(src + (c + u) * stride_c + 4 * g4);
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4) acc[g4] += x[u][g4];
    }
    for (; c < c1; ++c) {
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) acc[g4] += *reinterpret_cast<const f32x4 *>(src + c * stride_c + 4 * g4);
    }
    if (wave > 0) {
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) *reinterpret_cast<f32x4 *>(&red[wave - 1][lane * 16 + 4 * g4]) = acc[g4];
    }
    __syncthreads();
    if (wave != 0) return;
#pragma unroll
    for (int w = 0; w < 3; ++w)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) acc[g4] += *reinterpret_cast<const f32x4 *>(&red[w][lane * 16 + 4 * g4]);
    // lane (h, n) holds key kt*32 + n at queries qt*32 + krow(i, h)
    const int h = lane >> 5, n = lane & 31;
    const int key = kt * 32 + n;
    float *dst = dbias + ph * (int64_t)L * L;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int qi = qt * 32 + krow(i, h);
        if (qi < L && key < L) dst[(int64_t)qi * L + key] = acc[i / 4][i % 4];
    }
}

// query tiles whose dBias accumulators stay in registers (the rest go to LDS)
template <int D, int NKT> constexpr int kFusedNQR = NKT <= 4 ? NKT : 5;

template <int D, int NKT, bool HB, bool BV>
hipError_t launch_fused_t(const FusedArgs &fa, hipStream_t s) {
    const unsigned grid = (unsigned)((fa.n_units + 7) / 8 * 8);  // XCD-aware order; surplus workgroups exit
    hipLaunchKernelGGL((bwd_fused_kernel<D, NKT, HB, BV, kFusedNQR<D, NKT>>), dim3(grid), dim3(NKT * 64), 0, s, fa);
    return hipGetLastError();
}

// With a bias, the chunk's dBias accumulators (a whole [L, L] plane per
// workgroup) must fit beside the rest: every head dim up to 128 keys, and at
// 256 keys head_dim 8 with rows of whole 16-byte groups (three query tiles of
// accumulators in LDS).  Other shapes take the two-pass backward.
template <int D, int NKT>
constexpr bool kFusedBias = NKT <= 4 || D == 8;

template <int D, int NKT>
hipError_t launch_fused_n(const Problem &p, const FusedArgs &fa, hipStream_t s) {
    if (!fa.bias) return launch_fused_t<D, NKT, false, true>(fa, s);
    if constexpr (kFusedBias<D, NKT>) {
        if (p.L % 8 == 0) return launch_fused_t<D, NKT, true, true>(fa, s);
        if constexpr (NKT <= 4) return launch_fused_t<D, NKT, true, false>(fa, s);
    }
    return hipErrorInvalidValue;  // excluded by fused_bwd_supported
}

template <int D>
hipError_t launch_fused_d(const Problem &p, const FusedArgs &fa, hipStream_t s) {
    const int64_t nkt = (p.L + 31) / 32;
    if (nkt <= 1) return launch_fused_n<D, 1>(p, fa, s);
    if (nkt <= 2) return launch_fused_n<D, 2>(p, fa, s);
    if (nkt <= 4) return launch_fused_n<D, 4>(p, fa, s);
    return launch_fused_n<D, 8>(p, fa, s);
}

}  // namespace

bool fused_bwd_supported(const Problem &p, bool has_bias) {
    const int64_t nkt = (p.L + 31) / 32;
    if (p.dtype != 1 || p.D > 32 || nkt > 8) return false;  // (its LDS tiles hold up to 256 keys)
    if (!has_bias) return true;
    return nkt <= 4 || (p.D == 8 && p.L % 8 == 0);
}

// rows per chunk and chunk count of the fused backward: about 2048 waves in
// all, each chunk of a plane's rows one workgroup per head
void fused_bwd_chunks(const Problem &p, bool has_bias, int64_t *chunks, int64_t *rows_per_chunk) {
    const int64_t planes = has_bias ? p.N / p.rpb : p.N;
    const int64_t rpb = has_bias ? p.rpb : 1;
    const int64_t nqt = (p.L + 31) / 32;
    const int64_t waves = nqt <= 1 ? 1 : nqt <= 2 ? 2 : nqt <= 4 ? 4 : 8;
    int64_t c = 1;
    if (has_bias && planes > 0) {
        const int64_t want_wg = 2048 / waves;
        c = (want_wg + planes * p.H - 1) / (planes * p.H);
        if (c < 1) c = 1;
        if (c > rpb) c = rpb;
    }
    const int64_t g = rpb > 0 ? (rpb + c - 1) / c : 1;
    *rows_per_chunk = g;
    *chunks = rpb > 0 ? (rpb + g - 1) / g : 1;
}

size_t fused_bwd_partial_bytes(const Problem &p, int64_t chunks) {
    if (chunks <= 1) return 0;
    const int64_t nqt = (p.L + 31) / 32;
    return (size_t)(p.N / p.rpb) * (size_t)chunks * (size_t)p.H * (size_t)(nqt * nqt) * 1024u * 4u;
}

hipError_t launch_bwd_fused(const Problem &p, const BwdPtrs &x, void *ws, int64_t chunks, int64_t rows_per_chunk,
                            hipStream_t s, Tracer &tr) {
    FusedArgs fa;
    fa.q = x.q; fa.k = x.k; fa.v = x.v; fa.g = x.g; fa.out = x.out; fa.dout = x.dout; fa.bias = x.bias;
    fa.mask = x.mask; fa.lse = x.lse;
    fa.dq = x.dq; fa.dk = x.dk; fa.dv = x.dv; fa.dg = x.dg;
    fa.dbias = x.dbias;
    fa.part = (x.bias && chunks > 1) ? (float *)ws : nullptr;
    fa.L = p.L; fa.srow = p.srow; fa.stok = p.stok; fa.H = p.H;
    fa.scale = 1.0f / sqrtf((float)p.D);
    // without a bias every row is its own group
    fa.rpb = x.bias ? p.rpb : 1;
    fa.chunks = x.bias ? chunks : 1;
    fa.rows_per_chunk = x.bias ? rows_per_chunk : 1;
    const int64_t planes = x.bias ? p.N / p.rpb : p.N;
    fa.n_units = planes * fa.chunks * p.H;
    hipError_t e;
    switch (p.D) {
        case 8: e = launch_fused_d<8>(p, fa, s); break;
        case 16: e = launch_fused_d<16>(p, fa, s); break;
        default: e = launch_fused_d<32>(p, fa, s); break;
    }
    if (e != hipSuccess) return e;
    tr.mark(s);
    if (fa.part) {
        const int64_t nqt = (p.L + 31) / 32;
        const int64_t blocks = planes * p.H * nqt * nqt;
        hipLaunchKernelGGL(dbias_tiles_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                           (const float *)fa.part, x.dbias, planes, p.H, chunks, (int)p.L);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        tr.mark(s);
    }
    return hipSuccess;
}

}  // namespace evo
