// evo_fwd.hip -- forward kernel of the gated attention with pair bias, gfx950.
//
// o = sigmoid(g) * softmax(Q K^T / sqrt(d) + bias + mask) V, plus the
// per-query log-sum-exp (ScaleFold Section 3.3, "Multi Head Attention": the
// pair bias enters the logits before the softmax; all of MHA in one kernel).
//
// Work unit = one (row, head), one workgroup per unit, one wave per
// 32-query tile (at most 16 waves: 512 keys); at head_dim 64 a unit
// is a (row, head, half of the channels of O): both halves form the same
// logits from all 64 channels, each produces 32 channels of O, and the first
// writes the log-sum-exp.  The kernel keeps its
// registers low (about 90 at head_dim 32) so that two workgroups share a CU
// and each hides the other's loads and barriers.  K and V sit row-major in
// LDS; the V^T operand of O^T = V^T P^T comes out of the transposing LDS read
// (ds_read_b64_tr_b16) on the bf16 path.
//
// Logits are produced transposed (S^T = K Q^T): a lane owns one query and
// the keys sit in its registers, so row max and row sum are in-lane
// reductions plus one exchange between the two lane halves, and the
// probabilities in registers are already the B operand of O^T = V^T P^T.
//
// bf16 path, per key tile of 32 keys:
//   * the logits are kept "raw", S_raw = K Q^T + sqrt(d) * bias; the pair
//     bias enters through the MFMA accumulator: a constant A operand holding
//     sqrt(d) (split into two bf16 terms) on a permuted diagonal times the
//     bias row loaded as raw bf16 (the B operand) -- no per-logit unpacking;
//   * the scale 1/sqrt(d) and log2(e) are folded into the exponent's FMA;
//   * with head_dim < 32, a row of ones in the V^T operand makes the same
//     MFMA produce the row sums of the probabilities.
// The running max is only raised when a tile's max exceeds it by more than
// 2^8 in the base-2 exponent, so rescaling the accumulators is rare.
//
// Memory: every global access is a buffer instruction on a per-unit
// resource; out-of-range lanes get an out-of-range offset (zeros on load,
// dropped on store) instead of a branch.  All loads are therefore issued
// unconditionally, in the order they are needed (the next key tile's bias
// before the current tile's math), which keeps the compiler's in-order load
// counters exact.
#include <math.h>
#include <stdlib.h>

#include "evo_frag.h"
#include "evo_kernels.h"

namespace evo {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.69314718055994531f;

// Running-max policy: the reference max is raised only where a chunk max
// exceeds it by more than 2^kTau (base-2 exponent units), so unnormalised
// probabilities stay below 2^kTau.
constexpr float kTau = 8.0f;

struct FwdArgs {
    const void *q, *k, *v, *g, *bias;
    const uint8_t *mask;
    void *out;
    float *lse;
    int64_t L, rpb, srow, stok, n_units;
    int H;
    float scale;
};

// raw bf16 pair bias of key tile kt for query row qi, in the k32 slot order:
// slots {8h+s, 16+8h+s} = keys kt*32 + those slots.  Rows past L
// read zeros; keys past L read the next row's values (those keys are masked,
// so the values never matter).  BV: L % 8 == 0, rows are 16-byte aligned.
template <bool BV>
__device__ __forceinline__ Tr<bf16_t>::K32 bias_k32(rsrc_t rb, int qi, int kt, int L, int h) {
    Tr<bf16_t>::K32 f;
    const uint32_t e0 = (uint32_t)(qi * L + kt * 32 + 8 * h);  // element index of slot 0
    if constexpr (BV) {
        f.v[0] = __builtin_bit_cast(bf16x8, bload16(rb, e0 * 2u));
        f.v[1] = __builtin_bit_cast(bf16x8, bload16(rb, e0 * 2u + 32u));
    } else {
        short8tr w0, w1;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            w0[s] = (short)bload2(rb, (e0 + s) * 2u);
            w1[s] = (short)bload2(rb, (e0 + 16 + s) * 2u);
        }
        f.v[0] = __builtin_bit_cast(bf16x8, w0);
        f.v[1] = __builtin_bit_cast(bf16x8, w1);
    }
    return f;
}

// A bias fragment as the starting value of a logit tile: register i holds
// sqd * bias of key krow(i, h) -- the k32 slot order is the accumulator's
// register order -- in fp32, one rounding of the product.  Passed as the C
// operand of the tile's first QK^T product, it adds the scaled pair bias
// without any bias product on the matrix unit.
__device__ __forceinline__ f32x16 bias_acc(const Tr<bf16_t>::K32 &b, float sqd) {
    f32x16 c;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int s = 0; s < 8; ++s) c[8 * t + s] = sqd * (float)b.v[t][s];
    return c;
}

// 64-lane mask of the lanes whose logit register i belongs to a kept key:
// register i of lane half h holds key krow(i, h) of the tile.
__device__ __forceinline__ uint64_t key_lanes(uint32_t kb, int i) {
    const uint64_t lo = (kb >> krow(i, 0)) & 1u, hi = (kb >> krow(i, 1)) & 1u;
    return (lo ? 0x00000000ffffffffull : 0ull) | (hi ? 0xffffffff00000000ull : 0ull);
}

// QG: query groups per unit.  A unit's NKT query tiles run as QG workgroups
// of NKT / QG waves each (all of them stage the unit's K and V), so that a
// call with few (row, head) units still fills the chip.
template <typename T, int D, int NKT, int KC, bool BV, int QG>
__global__ void __launch_bounds__(NKT / QG * 64) fwd_kernel(FwdArgs a) {
    using E = typename Tr<T>::elem;
    using K32 = typename Tr<T>::K32;
    constexpr int ES = sizeof(E);
    constexpr bool kBf = ES == 2;              // bf16: V^T via the transposing LDS read, bias via MFMA
    // output channels per workgroup: head_dim 64 runs as two units per (row,
    // head), each contracting over all 64 channels for the logits and
    // producing 32 channels of O
    constexpr int DO = D > 32 ? 32 : D;
    constexpr int NHALF = D / DO;
    constexpr bool kOnesRow = kBf && DO < 32;  // row sums come out of the PV product
    constexpr int VEC = Tr<T>::VEC;
    constexpr int CPT = D / VEC;               // 16-byte chunks per token
    constexpr int LP = NKT * 32;
    constexpr int NW = NKT / QG;               // waves (query tiles) per workgroup
    constexpr int NT = NW * 64;
    constexpr int NKB = (LP + NT - 1) / NT;    // keys per thread for the mask bits
    constexpr int KSTR = D + VEC;              // row stride of K / V in LDS (elements)
    constexpr int VSTR = LP + VEC;             // row stride of V^T in LDS (fp32 path)
    // bf16: V rows in LDS are 32 columns wide whatever the head dim (the
    // unit's DO channels), the columns past DO holding constants (a 1 in column
    // DO when the row sums come from the PV product, zeros elsewhere), so the
    // transposing read needs no per-lane substitution
    constexpr int VSTRB = 32 + VEC;
    constexpr int PCH = (32 - DO) / 8;         // constant 16-byte chunks per V row
    constexpr int NCH = NKT / KC;              // chunks of KC key tiles
    constexpr int NPF = (LP * CPT + NT - 1) / NT;  // 16-byte chunks of K (and of V) per thread
    constexpr int NBB = kBf && BV ? KC : 1;    // bias fragments per chunk held in registers
    constexpr int NG = ES == 2 ? 1 : 2;        // 16-byte gate loads per 8 channels
    // bf16 at head_dim 8: the logit product runs on the k=16 instruction; each
    // K row in LDS is followed by its k-slots 8..15 (the key's masked-key word,
    // then zeros) and each query has a 1 in slot 8, so the product also adds
    // -2^64 on masked keys and no separate masked-key term is needed
    constexpr bool kPad8 = kBf && D == 8;
    using QKF = typename QKFragSel<T, D>::type;
    static_assert(!kPad8 || (CPT == 1 && NPF == NKB), "one K chunk and one mask byte per key and thread step");
    __shared__ __attribute__((aligned(16))) E k_lds[LP * KSTR];
    __shared__ __attribute__((aligned(16))) E v_lds[kBf ? LP * VSTRB : DO * VSTR];
    __shared__ uint32_t kbits[NKT];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h2 = lane >> 5, n = lane & 31;
    const int L = (int)a.L;
    // one workgroup per (row, head[, channel half], query group) unit;
    // consecutive units (the query groups and heads of a row) land on the
    // same XCD
    const int64_t u = xcd_unit(blockIdx.x, gridDim.x);
    if (u >= a.n_units) return;
    const int qg = QG == 1 ? 0 : (int)(u % QG);
    const int64_t uh = u / QG;
    const int qi = (qg * NW + wave) * 32 + n;
    const bool qvalid = qi < L;
    const bool has_bias = a.bias != nullptr, has_mask = a.mask != nullptr, has_gate = a.g != nullptr;
    const uint32_t stok_b = (uint32_t)(a.stok * ES);
    const uint32_t row_bytes = (uint32_t)(a.L * a.stok * ES);  // host: below 2^31
    const uint32_t q_off = qvalid ? (uint32_t)qi * stok_b : kOOB;

    const int ch = NHALF == 1 ? 0 : (int)(uh % NHALF);
    const int c_off = ch * DO;  // first output channel of the unit
    const int64_t r = uh / NHALF / a.H;
    const int hh = (int)(uh / NHALF % a.H);
    auto tok_buf = [&](const void *X) {
        return make_buf((const E *)X + r * a.srow + (int64_t)hh * D, row_bytes);
    };
    const rsrc_t rb = has_bias ? make_buf((const E *)a.bias + ((r / a.rpb) * a.H + hh) * (int64_t)L * L,
                                          (uint32_t)(L * L * ES))
                               : make_buf(nullptr, 0u);

    // ---- loads of the unit, in the order they are needed
    {
        const rsrc_t rk = tok_buf(a.k), rv = tok_buf(a.v);
        u32x4 kr[NPF], vr[NPF];
#pragma unroll
        for (int j = 0; j < NPF; ++j) {
            const int idx = tid + j * NT;
            const int t = idx / CPT, c = (idx % CPT) * VEC;
            const uint32_t off = (idx < LP * CPT && t < L) ? (uint32_t)t * stok_b + (uint32_t)(c * ES) : kOOB;
            kr[j] = bload16(rk, off);
            vr[j] = bload16(rv, off);
        }
        const rsrc_t rmask = has_mask ? make_buf(a.mask + r * a.L, (uint32_t)L) : make_buf(nullptr, 0u);
        uint32_t mb[NKB];
#pragma unroll
        for (int j = 0; j < NKB; ++j) mb[j] = bload1(rmask, (uint32_t)(tid + j * NT));
#pragma unroll
        for (int j = 0; j < NPF; ++j) {
            const int idx = tid + j * NT;
            if (idx < LP * CPT) {
                const int t = idx / CPT, c = (idx % CPT) * VEC;
                *reinterpret_cast<u32x4 *>(&k_lds[t * KSTR + c]) = kr[j];
                if constexpr (kPad8) {
                    const bool keep = (!has_mask || mb[j] != 0) && t < L;
                    const u32x4 w = {keep ? 0u : (uint32_t)(uint16_t)kBf16MaskNeg, 0u, 0u, 0u};
                    *reinterpret_cast<u32x4 *>(&k_lds[t * KSTR + 8]) = w;
                }
                const int cv = c - c_off;  // V: only the unit's output channels
                if (NHALF == 1 || (cv >= 0 && cv < DO)) {
                    if constexpr (kBf) {
                        *reinterpret_cast<u32x4 *>(&v_lds[t * VSTRB + cv]) = vr[j];
                    } else {
                        const E *ve = reinterpret_cast<const E *>(&vr[j]);
#pragma unroll
                        for (int e = 0; e < VEC; ++e) v_lds[(cv + e) * VSTR + t] = ve[e];
                    }
                }
            }
        }
        if constexpr (kBf && PCH > 0) {
            for (int idx = tid; idx < LP * PCH; idx += NT) {
                const int t = idx / PCH, pc = idx % PCH;
                const u32x4 w = {(pc == 0 && kOnesRow) ? (uint32_t)(uint16_t)kBf16One : 0u, 0u, 0u, 0u};
                *reinterpret_cast<u32x4 *>(&v_lds[t * VSTRB + DO + 8 * pc]) = w;
            }
        }
        // key-mask bits of every key tile: 64 keys per wave and step
#pragma unroll
        for (int j = 0; j < NKB; ++j) {
            const int key = tid + j * NT;
            const bool keep = (!has_mask || mb[j] != 0) && key < L;
            const unsigned long long bal = __ballot(keep);
            const int kt0 = (j * NT + wave * 64) / 32;
            if (lane == 0) {
                if (kt0 < NKT) kbits[kt0] = (uint32_t)bal;
                if (kt0 + 1 < NKT) kbits[kt0 + 1] = (uint32_t)(bal >> 32);
            }
        }
    }
    QKF qf;
    if constexpr (kPad8) qf.load(tok_buf(a.q), q_off, h2, kBf16One);
    else qf.load(tok_buf(a.q), q_off, h2);
    // bias of the first chunk, then the gate (needed last)
    K32 bcur[NBB];
    if constexpr (kBf && BV) {
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) bcur[kc] = bias_k32<BV>(rb, qi, kc, L, h2);
    }
    const rsrc_t rg = has_gate ? tok_buf(a.g) : make_buf(nullptr, 0u);
    u32x4 graw[2][NG];
#pragma unroll
    for (int half = 0; half < 2; ++half) {
        const int cb = 16 * half + 8 * h2;  // channels of O^T registers 8*half .. 8*half+7
        if (16 * half >= DO) continue;
        const uint32_t off = cb < DO ? q_off + (uint32_t)((c_off + cb) * ES) : kOOB;
#pragma unroll
        for (int gi = 0; gi < NG; ++gi) graw[half][gi] = bload16(rg, off + 16u * gi);
    }

    // logits are kept as K Q^T + sqrt(d) * bias ("raw" units); the softmax
    // scale 1/sqrt(d) and log2(e) are folded into the exponent
    const float c2 = a.scale * kLog2e;
    float sq_hi, sq_lo;
    sqrt_split(D, sq_hi, sq_lo);
    const float sqd = sq_hi + sq_lo;
    __syncthreads();

    float m2 = -INFINITY;  // reference max, base-2 exponent units (per query)
    float lsum = 0.0f;     // row sum (unused with the ones row)
    f32x16 o = zero16();
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        // ---- the next chunk's bias goes out first (loads complete in order)
        K32 bnext[NBB];
        if constexpr (kBf && BV) {
            if (c + 1 < NCH) {
#pragma unroll
                for (int kc = 0; kc < KC; ++kc) bnext[kc] = bias_k32<BV>(rb, qi, (c + 1) * KC + kc, L, h2);
            }
        }
        // ---- pass 1: raw logits of the chunk and their max
        f32x16 s[KC];
        uint32_t kbs[KC];
        float mx = -INFINITY;
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) {
            const int kt = c * KC + kc;
            // tiles whose bias is read per tile load it before any branch
            K32 bt;
            float bf[16];
            if constexpr (kBf && !BV) bt = bias_k32<false>(rb, qi, kt, L, h2);
            if constexpr (!kBf) {
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const uint32_t j = (uint32_t)(kt * 32 + krow(i, h2));
                    bf[i] = __builtin_bit_cast(float, bload4(rb, ((uint32_t)qi * L + j) * 4u));
                }
            }
            const uint32_t kb = __builtin_amdgcn_readfirstlane(kbits[kt]);
            kbs[kc] = kb;
            if (kb == 0) continue;
            QKF kf;
            kf.load(&k_lds[(kt * 32 + sig(n)) * KSTR], h2);
            s[kc] = zero16();
            if constexpr (kBf) {
                if constexpr (BV) bt = bcur[kc];
                if (has_bias) s[kc] = bias_acc(bt, sqd);
            }
            QKF::mma(s[kc], kf, qf);
            if constexpr (!kBf) {
                if (has_bias) {
#pragma unroll
                    for (int i = 0; i < 16; ++i) s[kc][i] = __builtin_fmaf(bf[i], sqd, s[kc][i]);
                }
            }
            if (kb != 0xffffffffu) {
                if constexpr (kPad8) {
                    // the masked-key term came with the product
                } else if constexpr (kBf) {
                    // masked keys: -2^64 on their rows (row n of the tile is key sig(n))
                    const short mv = ((kb >> sig(n)) & 1u) ? (short)0 : kBf16MaskNeg;
                    mma_rank1(s[kc], mv, kBf16One, h2);
                } else {
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        s[kc][i] = __builtin_amdgcn_inverse_ballot_w64(key_lanes(kb, i)) ? s[kc][i] : -INFINITY;
                }
            }
#pragma unroll
            for (int i = 0; i < 16; i += 2) mx = fmaxf(mx, fmaxf(s[kc][i], s[kc][i + 1]));
        }
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float mxl = mx * c2;
        // raise the reference max only where a chunk max exceeds it by more
        // than 2^kTau (always at the first finite max)
        const bool need = mxl > m2 + kTau;
        if (__ballot(need)) {
            const float alpha = need ? (m2 == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(m2 - mxl)) : 1.0f;
            if (need) m2 = mxl;
            lsum *= alpha;
#pragma unroll
            for (int i = 0; i < 16; ++i) o[i] *= alpha;
        }
        // a query whose keys so far are all masked keeps o = 0
        const float m2e = (m2 == -INFINITY) ? 0.0f : m2;
        // ---- pass 2: probabilities (unnormalised), row sum, O^T += V^T P^T
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) {
            const int kt = c * KC + kc;
            if (kbs[kc] == 0) continue;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kc][i], c2, -m2e));
                s[kc][i] = p;
                if constexpr (!kOnesRow) lsum += p;
            }
            const K32 pb = Tr<T>::pack(s[kc]);
            K32 va;
            if constexpr (kBf) {
                va = load_k32_tr(v_lds, VSTRB, kt * 32, 32, lane);
            } else {
                if (sig(n) < DO) va = load_k32<T>(&v_lds[sig(n) * VSTR + kt * 32], h2);
                else va = zero_k32<T>();
            }
            Tr<T>::mma_k32(o, va, pb);
        }
        if constexpr (kBf && BV) {
            if (c + 1 < NCH) {
#pragma unroll
                for (int kc = 0; kc < KC; ++kc) bcur[kc] = bnext[kc];
            }
        }
    }
    if constexpr (kOnesRow) {
        // channel D of O^T is the row sum: register 8*(D/16) + D%8 of lane half (D/8)%2
        constexpr int ri = 8 * (DO / 16) + DO % 8, rh = (DO / 8) % 2;
        const float own = o[ri], other = __shfl_xor(own, 32);
        lsum = (h2 == rh) ? own : other;
    } else {
        lsum += __shfl_xor(lsum, 32);
    }

    // ---- epilogue: normalise, gate, store O and lse (out-of-range lanes
    // store to an out-of-range offset, which is dropped)
    const float inv = lsum > 0.0f ? __builtin_amdgcn_rcpf(lsum) : 0.0f;
    const rsrc_t ro = tok_buf(a.out);
#pragma unroll
    for (int half = 0; half < 2; ++half) {
        const int cb = 16 * half + 8 * h2;
        if (16 * half >= DO) continue;
        const uint32_t off = cb < DO ? q_off + (uint32_t)((c_off + cb) * ES) : kOOB;
        float gv[8];
        if constexpr (ES == 2) {
            const u32x4 w = graw[half][0];
            const uint32_t ws[4] = {w.x, w.y, w.z, w.w};  // integer components (no bit_cast of a component)
#pragma unroll
            for (int s2 = 0; s2 < 4; ++s2) {
                gv[2 * s2] = __builtin_bit_cast(float, ws[s2] << 16);
                gv[2 * s2 + 1] = __builtin_bit_cast(float, ws[s2] & 0xffff0000u);
            }
        } else {
#pragma unroll
            for (int gi = 0; gi < NG; ++gi) {
                const f32x4 w = __builtin_bit_cast(f32x4, graw[half][gi]);
                gv[4 * gi] = w.x; gv[4 * gi + 1] = w.y; gv[4 * gi + 2] = w.z; gv[4 * gi + 3] = w.w;
            }
        }
        float val[8];
#pragma unroll
        for (int s8 = 0; s8 < 8; ++s8) {
            const float sg = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-gv[s8] * kLog2e));
            val[s8] = o[8 * half + s8] * inv * (has_gate ? sg : 1.0f);
        }
        if constexpr (ES == 2) {
            u32x4 w;
            w.x = (uint32_t)f2bf(val[0]) | ((uint32_t)f2bf(val[1]) << 16);
            w.y = (uint32_t)f2bf(val[2]) | ((uint32_t)f2bf(val[3]) << 16);
            w.z = (uint32_t)f2bf(val[4]) | ((uint32_t)f2bf(val[5]) << 16);
            w.w = (uint32_t)f2bf(val[6]) | ((uint32_t)f2bf(val[7]) << 16);
            bstore16(w, ro, off);
        } else {
            const f32x4 w0 = {val[0], val[1], val[2], val[3]}, w1 = {val[4], val[5], val[6], val[7]};
            bstore16(__builtin_bit_cast(u32x4, w0), ro, off);
            bstore16(__builtin_bit_cast(u32x4, w1), ro, off + 16u);
        }
    }
    // lse in natural-log units: (m2 + log2 lsum) * ln 2
    const float lse = lsum > 0.0f ? (m2 + __builtin_amdgcn_logf(lsum)) * kLn2 : -INFINITY;
    bstore4(__builtin_bit_cast(uint32_t, lse), make_buf(a.lse + (r * a.H + hh) * a.L, (uint32_t)L * 4u),
            (h2 == 0 && qvalid && ch == 0) ? (uint32_t)qi * 4u : kOOB);
}

// ---------------------------------------------------------------------------
// Row-walking forward for a pair bias shared by all rows (bf16, head_dim <=
// 32, at most 256 keys).  A fixed grid of workgroups, its size a multiple of
// the head count, walks the units u, u + G, u + 2G, ... (G = grid size): all
// units of a workgroup are rows of one head under the one bias plane.  Each
// wave loads its query tile's bias rows once and keeps them in registers as
// the fp32 starting values of its logit tiles (sqrt(d) * bias, 128 registers
// at 256 keys), reused for every row it visits, so the pair bias leaves L2
// once per workgroup instead of once per (row, head).  The next unit's K, V,
// key mask and query tile are requested during the current unit's first key
// tile and held in registers until that unit is staged; the gate during the
// last key tile; each key tile reads the next tile's K and V^T operands and
// mask word from LDS before its own math.  The constant columns of the V tile
// are set up once per workgroup.  Per key tile, against the one-unit kernel
// above: the masked-key operand is one LDS word (written at staging; at
// head_dim 8 it rides in the logit product's spare k-slots, as in the one-unit
// kernel), the tile max is a chain of three-input maxima,
// the two lane halves exchange their maxima only when some lane's own
// maximum calls for a raise of the reference max (no lane's own maximum
// above the threshold means no combined one is), and the exponent offset
// changes only with that max.  Every value is computed as in the one-unit
// kernel: the outputs are the same bits.
template <int D, int NKT>
__global__ void __launch_bounds__(NKT * 64) __attribute__((amdgpu_waves_per_eu(2))) fwd_rows_kernel(FwdArgs a) {
    using T = bf16_t;
    using E = uint16_t;
    using K32 = Tr<bf16_t>::K32;
    static_assert(D == 8 || D == 16 || D == 32, "bf16 head_dim up to 32");
    static_assert(NKT <= 8, "bias rows of up to 256 keys in registers");
    constexpr int VEC = 8;
    constexpr int CPT = D / VEC;               // 16-byte chunks per token
    constexpr int LP = NKT * 32;
    constexpr int NT = NKT * 64;               // two threads per key: one key-mask byte each suffices
    constexpr int KSTR = D + VEC;              // row stride of K in LDS (elements)
    constexpr int VSTRB = 32 + VEC;            // V rows: 32 columns (data, then constants), padded
    constexpr int PCH = (32 - D) / 8;          // constant 16-byte chunks per V row
    constexpr bool kOnesRow = D < 32;          // row sums come out of the PV product
    constexpr int NPF = (LP * CPT + NT - 1) / NT;
    // head_dim 8: the logit product on the k=16 instruction, the masked-key
    // word in each K row's slot 8 (as in the one-unit kernel)
    constexpr bool kPad8 = D == 8;
    using QKF = typename QKFragSel<T, D>::type;
    static_assert(!kPad8 || NPF == 1, "one K chunk per key, staged by the thread of that key");
    __shared__ __attribute__((aligned(16))) E k_lds[LP * KSTR];
    __shared__ __attribute__((aligned(16))) E v_lds[LP * VSTRB];
    __shared__ uint32_t mneg_lds[LP];          // masked-key operand per key: -2^64 (bf16, low half) or 0
    __shared__ uint32_t kbits[NKT];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h2 = lane >> 5, n = lane & 31;
    const int L = (int)a.L;
    const int qi = wave * 32 + n;
    const bool qvalid = qi < L;
    const bool has_mask = a.mask != nullptr, has_gate = a.g != nullptr;
    const uint32_t stok_b = (uint32_t)(a.stok * 2);
    const uint32_t row_bytes = (uint32_t)(a.L * a.stok * 2);  // host: below 2^31
    const uint32_t q_off = qvalid ? (uint32_t)qi * stok_b : kOOB;
    const rsrc_t none = make_buf(nullptr, 0u);

    // ---- per-workgroup constants
    const float c2 = a.scale * kLog2e;
    float sq_hi, sq_lo;
    sqrt_split(D, sq_hi, sq_lo);
    const float sqd = sq_hi + sq_lo;
    // B operand of the masked-key term: 1 in k-slot 0 (lane half 0), zeros
    // elsewhere, so only the A operand's slot 0 (the key's mask word) counts
    const short4v mask_b = {h2 == 0 ? kBf16One : (short)0, 0, 0, 0};
    if constexpr (PCH > 0) {
        for (int idx = tid; idx < LP * PCH; idx += NT) {
            const int t = idx / PCH, pc = idx % PCH;
            const u32x4 w = {(pc == 0 && kOnesRow) ? (uint32_t)(uint16_t)kBf16One : 0u, 0u, 0u, 0u};
            *reinterpret_cast<u32x4 *>(&v_lds[t * VSTRB + D + 8 * pc]) = w;
        }
    }

    // unit u -> (row ur, head uh), advanced incrementally: u grows by G per step
    const int H = a.H;
    const int64_t G = gridDim.x;
    const int64_t GH = G / H;
    const int Gh = (int)(G % H);  // 0: the host makes G a multiple of H
    int64_t u = xcd_unit(blockIdx.x, G);
    int64_t ur = u / H;
    int uh = (int)(u % H);
    // first element of a unit's [L, d] block in the token tensors; a unit past
    // the last one gets an empty resource (its loads read zeros)
    auto tok_buf = [&](const void *X, int64_t tb, bool ok) {
        return make_buf((const E *)X + (ok ? tb : 0), ok ? row_bytes : 0u);
    };

    // ---- this wave's bias rows (query tile `wave`, every key tile), once;
    // the host guarantees a single plane: plane 0 for every row.  They are
    // kept as the fp32 starting values of the logit tiles (sqrt(d) * bias)
    f32x16 bacc[NKT];
    {
        const rsrc_t rb = u < a.n_units ? make_buf((const E *)a.bias + (int64_t)uh * L * L, (uint32_t)(L * L * 2))
                                        : none;
#pragma unroll
        for (int kt = 0; kt < NKT; ++kt) bacc[kt] = bias_acc(bias_k32<true>(rb, qi, kt, L, h2), sqd);
    }

    // ---- the in-flight unit's K, V, key-mask byte and query tile
    u32x4 kr[NPF], vr[NPF];
    uint32_t mr;
    QKF qn;
    auto issue_unit = [&](int64_t rr, int h, bool ok) {
        const int64_t tb = rr * a.srow + (int64_t)h * D;
        const rsrc_t rk = tok_buf(a.k, tb, ok), rv = tok_buf(a.v, tb, ok);
#pragma unroll
        for (int j = 0; j < NPF; ++j) {
            const int idx = tid + j * NT;
            const int t = idx / CPT, c = (idx % CPT) * VEC;
            const uint32_t off = (idx < LP * CPT && t < L) ? (uint32_t)t * stok_b + (uint32_t)(c * 2) : kOOB;
            kr[j] = bload16(rk, off);
            vr[j] = bload16(rv, off);
        }
        const rsrc_t rm = (has_mask && ok) ? make_buf(a.mask + rr * a.L, (uint32_t)L) : none;
        mr = bload1(rm, (uint32_t)tid);
        if constexpr (kPad8) qn.load(tok_buf(a.q, tb, ok), q_off, h2, kBf16One);
        else qn.load(tok_buf(a.q, tb, ok), q_off, h2);
    };

    // every load is issued whether or not a mask or gate exists (an empty
    // resource reads zeros): a load behind a branch would leave the
    // compiler's in-order load counters unknown after the join, and it would
    // then wait for every load in flight, prefetches included
    issue_unit(ur, uh, u < a.n_units);
    for (; u < a.n_units; u += G) {
        const int64_t tb = ur * a.srow + (int64_t)uh * D;
        int64_t rn = ur + GH;
        int hn = uh + Gh;
        if (hn >= H) { hn -= H; ++rn; }
        const bool okn = u + G < a.n_units;
        __syncthreads();  // the previous unit's reads of the LDS tiles are done
        // ---- stage the unit: registers -> LDS, key-mask words and bits
        const bool keep = (!has_mask || mr != 0) && tid < L;  // key tid
#pragma unroll
        for (int j = 0; j < NPF; ++j) {
            const int idx = tid + j * NT;
            if (idx < LP * CPT) {
                const int t = idx / CPT, c = (idx % CPT) * VEC;
                *reinterpret_cast<u32x4 *>(&k_lds[t * KSTR + c]) = kr[j];
                *reinterpret_cast<u32x4 *>(&v_lds[t * VSTRB + c]) = vr[j];
                if constexpr (kPad8) {  // t == tid
                    const u32x4 w = {keep ? 0u : (uint32_t)(uint16_t)kBf16MaskNeg, 0u, 0u, 0u};
                    *reinterpret_cast<u32x4 *>(&k_lds[t * KSTR + 8]) = w;
                }
            }
        }
        {
            if constexpr (!kPad8) {
                if (tid < LP) mneg_lds[tid] = keep ? 0u : (uint32_t)(uint16_t)kBf16MaskNeg;
            }
            const unsigned long long bal = __ballot(keep);
            if (lane == 0) {
                if (2 * wave < NKT) kbits[2 * wave] = (uint32_t)bal;
                if (2 * wave + 1 < NKT) kbits[2 * wave + 1] = (uint32_t)(bal >> 32);
            }
        }
        const QKF qf = qn;
        __syncthreads();

        u32x4 graw = {0u, 0u, 0u, 0u}, graw2 = {0u, 0u, 0u, 0u};
        float m2 = -INFINITY;  // reference max, base-2 exponent units (per query)
        float nm2 = 0.0f;      // exponent offset: -m2 once m2 is finite
        float lsum = 0.0f;     // row sum (head_dim 32: no ones row)
        f32x16 o = zero16();
        // the unit's key-tile mask words, and the first tile's LDS operands;
        // each tile then reads the next tile's operands before its own math
        uint32_t kbs[NKT];
#pragma unroll
        for (int kt = 0; kt < NKT; ++kt) kbs[kt] = __builtin_amdgcn_readfirstlane(kbits[kt]);
        QKF kf_n;
        kf_n.load(&k_lds[sig(n) * KSTR], h2);
        uint32_t mw_n = kPad8 ? 0u : mneg_lds[sig(n)];
        K32 va_n = load_k32_tr(v_lds, VSTRB, 0, 32, lane);
#pragma unroll
        for (int kt = 0; kt < NKT; ++kt) {
            const QKF kf = kf_n;
            const uint32_t mwv = mw_n;
            const K32 va = va_n;
            if (kt + 1 < NKT) {
                kf_n.load(&k_lds[((kt + 1) * 32 + sig(n)) * KSTR], h2);
                if constexpr (!kPad8) mw_n = mneg_lds[(kt + 1) * 32 + sig(n)];
                va_n = load_k32_tr(v_lds, VSTRB, (kt + 1) * 32, 32, lane);
            }
            // ---- global loads, in the order they are waited for
            if (kt == 0) issue_unit(rn, hn, okn);
            if (kt == NKT - 1) {
                const rsrc_t rg = has_gate ? tok_buf(a.g, tb, true) : none;
                graw = bload16(rg, 8 * h2 < D ? q_off + (uint32_t)(8 * h2 * 2) : kOOB);
                if constexpr (D > 16) graw2 = bload16(rg, q_off + (uint32_t)((16 + 8 * h2) * 2));
            }
            const uint32_t kb = kbs[kt];
            if (kb != 0) {
                f32x16 s = bacc[kt];
                QKF::mma(s, kf, qf);
                if (!kPad8 && kb != 0xffffffffu) {
                    // masked keys: -2^64 on their rows (row n of the tile is key sig(n))
                    const u32x2 mw = {mwv, 0u};
                    s = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(__builtin_bit_cast(short4v, mw), mask_b, s, 0, 0, 0);
                }
                float mx = fmaxf(fmaxf(s[0], s[1]), s[2]);
#pragma unroll
                for (int i = 3; i < 15; i += 2) mx = fmaxf(fmaxf(mx, s[i]), s[i + 1]);
                mx = fmaxf(mx, s[15]);
                // raise the reference max only where the tile max exceeds it by
                // more than 2^kTau (always at the first finite max)
                if (__ballot(mx * c2 > m2 + kTau)) {
                    const float mxl = fmaxf(mx, __shfl_xor(mx, 32)) * c2;
                    const bool need = mxl > m2 + kTau;
                    const float alpha = need ? (m2 == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(m2 - mxl)) : 1.0f;
                    if (need) m2 = mxl;
                    nm2 = (m2 == -INFINITY) ? 0.0f : -m2;
                    lsum *= alpha;
#pragma unroll
                    for (int i = 0; i < 16; ++i) o[i] *= alpha;
                }
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[i], c2, nm2));
                    s[i] = p;
                    if constexpr (!kOnesRow) lsum += p;
                }
                const K32 pb = Tr<T>::pack(s);
                Tr<T>::mma_k32(o, va, pb);
            }
        }
        if constexpr (kOnesRow) {
            // channel D of O^T is the row sum: register 8*(D/16) + D%8 of lane half (D/8)%2
            constexpr int ri = 8 * (D / 16) + D % 8, rh = (D / 8) % 2;
            const float own = o[ri], other = __shfl_xor(own, 32);
            lsum = (h2 == rh) ? own : other;
        } else {
            lsum += __shfl_xor(lsum, 32);
        }

        // ---- epilogue: normalise, gate, store O and lse
        const float inv = lsum > 0.0f ? __builtin_amdgcn_rcpf(lsum) : 0.0f;
        const rsrc_t ro = tok_buf(a.out, tb, true);
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int cb = 16 * half + 8 * h2;
            if (16 * half >= D) continue;
            const uint32_t off = cb < D ? q_off + (uint32_t)(cb * 2) : kOOB;
            const u32x4 w = half == 0 ? graw : graw2;
            const uint32_t ws[4] = {w.x, w.y, w.z, w.w};  // integer components (no bit_cast of a component)
            float val[8];
#pragma unroll
            for (int s2 = 0; s2 < 4; ++s2) {
                const float g0 = __builtin_bit_cast(float, ws[s2] << 16);
                const float g1 = __builtin_bit_cast(float, ws[s2] & 0xffff0000u);
                const float sg0 = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-g0 * kLog2e));
                const float sg1 = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-g1 * kLog2e));
                val[2 * s2] = o[8 * half + 2 * s2] * inv * (has_gate ? sg0 : 1.0f);
                val[2 * s2 + 1] = o[8 * half + 2 * s2 + 1] * inv * (has_gate ? sg1 : 1.0f);
            }
            u32x4 wo;
            wo.x = (uint32_t)f2bf(val[0]) | ((uint32_t)f2bf(val[1]) << 16);
            wo.y = (uint32_t)f2bf(val[2]) | ((uint32_t)f2bf(val[3]) << 16);
            wo.z = (uint32_t)f2bf(val[4]) | ((uint32_t)f2bf(val[5]) << 16);
            wo.w = (uint32_t)f2bf(val[6]) | ((uint32_t)f2bf(val[7]) << 16);
            bstore16(wo, ro, off);
        }
        // lse in natural-log units: (m2 + log2 lsum) * ln 2
        const float lse = lsum > 0.0f ? (m2 + __builtin_amdgcn_logf(lsum)) * kLn2 : -INFINITY;
        bstore4(__builtin_bit_cast(uint32_t, lse), make_buf(a.lse + (ur * H + uh) * a.L, (uint32_t)L * 4u),
                (h2 == 0 && qvalid) ? (uint32_t)qi * 4u : kOOB);
        ur = rn;
        uh = hn;
    }
}

// key tiles per register-resident chunk: one keeps the kernel near 90
// registers (two tiles need about 130, which halves the occupancy)
template <int NKT> constexpr int kFwdKC = 1;

template <typename T, int D, int NKT, bool BV, int QG>
hipError_t launch_q(const Problem &p, const FwdPtrs &x, hipStream_t s) {
    // unaligned bias rows are read per element, one tile per chunk
    constexpr int KC = BV ? kFwdKC<NKT> : 1;
    FwdArgs a;
    a.q = x.q; a.k = x.k; a.v = x.v; a.g = x.g; a.bias = x.bias; a.mask = x.mask;
    a.out = x.out; a.lse = x.lse;
    a.L = p.L; a.rpb = p.rpb; a.srow = p.srow; a.stok = p.stok; a.H = p.H;
    a.n_units = p.N * p.H * (D > 32 ? D / 32 : 1) * QG;
    a.scale = 1.0f / sqrtf((float)D);
    // one workgroup per unit; the grid is rounded up to a multiple of 8 so
    // that the XCD-aware unit order applies (surplus workgroups exit)
    const int64_t nwg = (a.n_units + 7) / 8 * 8;
    hipLaunchKernelGGL((fwd_kernel<T, D, NKT, KC, BV, QG>), dim3((unsigned)nwg), dim3(NKT / QG * 64), 0, s, a);
    return hipGetLastError();
}

// Row-walking kernel: eligible when every row uses one bias plane, rows are
// 16-byte aligned (bf16, L % 8 == 0), at most 256 keys, and there are at
// least two units per resident workgroup (one 8-wave workgroup per CU at
// the kernel's two waves per SIMD: 256 CUs x 8 waves); with one, the bias
// held in registers would not be reused at all.  EVO_ATTN_FWD_ROWS=0
// in the environment at the time of the call selects the one-unit kernel
// instead (same results; read on every call, no state kept).
constexpr int64_t kRowsResidentWaves = 256 * 8;

inline bool fwd_rows_enabled() {
    const char *e = getenv("EVO_ATTN_FWD_ROWS");
    return !(e && e[0] == '0');
}

template <int D, int NKT>
hipError_t launch_rows(const Problem &p, const FwdPtrs &x, hipStream_t s, int64_t g) {
    FwdArgs a;
    a.q = x.q; a.k = x.k; a.v = x.v; a.g = x.g; a.bias = x.bias; a.mask = x.mask;
    a.out = x.out; a.lse = x.lse;
    a.L = p.L; a.rpb = p.rpb; a.srow = p.srow; a.stok = p.stok; a.H = p.H;
    a.n_units = p.N * p.H;
    a.scale = 1.0f / sqrtf((float)D);
    hipLaunchKernelGGL((fwd_rows_kernel<D, NKT>), dim3((unsigned)g), dim3(NKT * 64), 0, s, a);
    return hipGetLastError();
}

// Query groups per (row, head): with fewer units than two per CU (512), a
// unit's query tiles are split over two workgroups, over four at 64 units or
// fewer (each stages the unit's K and V, mostly from the L2 its XCD shares
// with the unit's other groups; at 128 units two were faster than four).
template <typename T, int D, int NKT, bool BV>
hipError_t launch_t(const Problem &p, const FwdPtrs &x, hipStream_t s) {
    const int64_t units = p.N * p.H * (D > 32 ? D / 32 : 1);
    if constexpr (sizeof(typename Tr<T>::elem) == 2 && D <= 32 && BV && NKT <= 8) {
        // grid: the resident workgroups, a multiple of 8 (XCD-aware order)
        // and of the head count (every workgroup keeps one head)
        const int64_t g0 = kRowsResidentWaves / NKT;
        const int64_t g = g0 / 8 / p.H * 8 * p.H;
        if (x.bias != nullptr && p.rpb >= p.N && g > 0 && units >= 2 * g0 && p.N < (int64_t(1) << 31) &&
            fwd_rows_enabled())
            return launch_rows<D, NKT>(p, x, s, g);
    }
    if constexpr (NKT >= 4) {
        if (units <= 64) return launch_q<T, D, NKT, BV, 4>(p, x, s);
        if (units < 512) return launch_q<T, D, NKT, BV, 2>(p, x, s);
    }
    return launch_q<T, D, NKT, BV, 1>(p, x, s);
}

template <typename T, int D, int NKT>
hipError_t launch_t(const Problem &p, const FwdPtrs &x, hipStream_t s) {
    // fp32 reads its bias per element either way
    if (sizeof(typename Tr<T>::elem) == 2 && p.L % Tr<T>::VEC == 0) return launch_t<T, D, NKT, true>(p, x, s);
    return launch_t<T, D, NKT, false>(p, x, s);
}

template <typename T, int D>
hipError_t launch_d(const Problem &p, const FwdPtrs &x, hipStream_t s) {
    const int64_t nkt = (p.L + 31) / 32;
    if (nkt <= 1) return launch_t<T, D, 1>(p, x, s);
    if (nkt <= 2) return launch_t<T, D, 2>(p, x, s);
    if (nkt <= 4) return launch_t<T, D, 4>(p, x, s);
    if (nkt <= 8) return launch_t<T, D, 8>(p, x, s);
    // 257..512 keys: 16 query tiles, 16 waves (bf16, head_dim <= 32: K and V
    // of 512 keys fit the LDS; the ABI rejects the rest before this point)
    if constexpr (sizeof(typename Tr<T>::elem) == 2 && D <= 32) return launch_t<T, D, 16>(p, x, s);
    else return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_dt(const Problem &p, const FwdPtrs &x, hipStream_t s) {
    switch (p.D) {
        case 8: return launch_d<T, 8>(p, x, s);
        case 16: return launch_d<T, 16>(p, x, s);
        case 64: return launch_d<T, 64>(p, x, s);
        default: return launch_d<T, 32>(p, x, s);
    }
}

}  // namespace

hipError_t launch_fwd(const Problem &p, const FwdPtrs &x, hipStream_t s) {
    if (p.dtype == 1) return launch_dt<bf16_t>(p, x, s);
    return launch_dt<float>(p, x, s);
}

}  // namespace evo
