// evo_fwd.hip -- forward kernel of the gated attention with pair bias, gfx950.
//
// o = sigmoid(g) * softmax(Q K^T / sqrt(d) + bias + mask) V, plus the
// per-query log-sum-exp (ScaleFold Section 3.3, "Multi Head Attention": the
// pair bias enters the logits before the softmax; all of MHA in one kernel).
//
// One workgroup owns one (row, head): it stages K (row-major) and V^T into
// LDS once, and each wave takes 32-query tiles.  A wave holds the logits of
// 128 keys (4 tiles of 32) in registers at a time, takes their max and
// exponentials in two passes over registers, and rescales its running sums
// between such chunks (once at seq_len 256).  Logits are produced transposed (S^T = K Q^T): a lane owns one
// query and the keys sit in its registers, so the row max and row sum are
// in-lane reductions plus one exchange between the two lane halves, and the
// probabilities in registers are already the B operand of O^T = V^T P^T.
#include <math.h>

#include "evo_frag.h"
#include "evo_kernels.h"

namespace evo {

namespace {

constexpr float kLog2e = 1.4426950408889634f;

struct FwdArgs {
    const void *q, *k, *v, *g, *bias;
    const uint8_t *mask;
    void *out;
    float *lse;
    int64_t L, rpb, srow, stok;
    int H;
    float scale;
};

// 8 consecutive bias values (keys j0..j0+7) of one query row as fp32;
// keys at or beyond L read as 0 (they are masked).
template <typename T>
__device__ __forceinline__ void load_bias8(const typename Tr<T>::elem *row, int j0, int L, bool vec_ok,
                                           float *out8) {
    using E = typename Tr<T>::elem;
    if (vec_ok && j0 + 8 <= L) {
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
        for (int s = 0; s < 8; ++s) out8[s] = (j0 + s < L) ? Tr<T>::to_f(row[j0 + s]) : 0.0f;
    }
}

template <typename T, int D, int NKT>
__global__ void __launch_bounds__(256) fwd_kernel(FwdArgs a) {
    using E = typename Tr<T>::elem;
    constexpr int VEC = Tr<T>::VEC;
    constexpr int LP = NKT * 32;        // keys rounded up to whole tiles
    constexpr int KSTR = D + VEC;       // K row stride in LDS (elements)
    constexpr int VSTR = LP + VEC;      // V^T row stride in LDS
    constexpr int NW = NKT < 4 ? NKT : 4;
    constexpr int NT = NW * 64;
    constexpr int KC = NKT < 4 ? NKT : 4;  // key tiles per register-resident chunk
    __shared__ __attribute__((aligned(16))) E k_lds[LP * KSTR];
    __shared__ __attribute__((aligned(16))) E vt_lds[D * VSTR];
    __shared__ uint32_t kbits[NKT];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h2 = lane >> 5, n = lane & 31;
    const int64_t unit = xcd_unit(blockIdx.x, gridDim.x);
    const int64_t r = unit / a.H;
    const int hh = (int)(unit % a.H);
    const int L = (int)a.L;
    const int64_t base = r * a.srow + (int64_t)hh * D;
    const E *Q = (const E *)a.q + base;
    const E *K = (const E *)a.k + base;
    const E *V = (const E *)a.v + base;

    // ---- stage K (row-major) and V^T into LDS; rows >= L are zero
    for (int idx = tid; idx < LP * (D / VEC); idx += NT) {
        const int t = idx / (D / VEC), c = (idx % (D / VEC)) * VEC;
        uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
        if (t < L) {
            kv = *reinterpret_cast<const uint4 *>(K + (int64_t)t * a.stok + c);
            vv = *reinterpret_cast<const uint4 *>(V + (int64_t)t * a.stok + c);
        }
        *reinterpret_cast<uint4 *>(&k_lds[t * KSTR + c]) = kv;
        const E *ve = reinterpret_cast<const E *>(&vv);
#pragma unroll
        for (int e = 0; e < VEC; ++e) vt_lds[(c + e) * VSTR + t] = ve[e];
    }
    // ---- key-keep bits, one 32-bit word per key tile
    {
        const int t = tid;  // NT >= LP
        bool keep = t < L;
        if (keep && a.mask) keep = a.mask[r * a.L + t] != 0;
        const unsigned long long bal = __ballot(keep);
        if (lane == 0) {
            if (2 * wave < NKT) kbits[2 * wave] = (uint32_t)bal;
            if (2 * wave + 1 < NKT) kbits[2 * wave + 1] = (uint32_t)(bal >> 32);
        }
    }
    __syncthreads();

    const E *bias_plane = nullptr;
    if (a.bias) bias_plane = (const E *)a.bias + ((r / a.rpb) * a.H + hh) * (int64_t)L * L;
    const bool bias_vec_ok = (L % VEC) == 0;
    const int nqt = (L + 31) / 32;

    for (int qt = wave; qt < nqt; qt += NW) {
        const int qi = qt * 32 + n;
        const bool qvalid = qi < L;
        ChFrag<T, D> qf;
        if (qvalid) qf.load(Q + (int64_t)qi * a.stok, h2);
        else qf.zero();

        // Keys are processed in chunks of KC tiles (128 keys); within a chunk
        // the logits stay in registers, between chunks the running max is
        // updated and the partial sums rescaled (one rescale at L = 256).
        float m_run = -INFINITY, lsum = 0.0f;
        f32x16 o = zero16();
        const int vrow = sig(n);
#pragma unroll
        for (int c0 = 0; c0 < NKT; c0 += KC) {
            // ---- pass 1: logits of the chunk and its max
            f32x16 s[KC];
            float mx = -INFINITY;
#pragma unroll
            for (int kc = 0; kc < KC; ++kc) {
                const int kt = c0 + kc;
                const uint32_t kb = __builtin_amdgcn_readfirstlane(kbits[kt]);  // wave-uniform
                if (kb == 0) continue;
                ChFrag<T, D> kf;
                kf.load(&k_lds[(kt * 32 + sig(n)) * KSTR], h2);
                s[kc] = zero16();
                ChFrag<T, D>::mma(s[kc], kf, qf);
                float b[16];
                if (bias_plane && qvalid) {
                    const E *brow = bias_plane + (int64_t)qi * L;
                    load_bias8<T>(brow, kt * 32 + 8 * h2, L, bias_vec_ok, b);
                    load_bias8<T>(brow, kt * 32 + 16 + 8 * h2, L, bias_vec_ok, b + 8);
                } else {
#pragma unroll
                    for (int i = 0; i < 16; ++i) b[i] = 0.0f;
                }
                const bool full = kb == 0xffffffffu;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    float t = __builtin_fmaf(s[kc][i], a.scale, b[i]);
                    if (!full && !((kb >> krow(i, h2)) & 1u)) t = -INFINITY;
                    s[kc][i] = t;
                    mx = fmaxf(mx, t);
                }
            }
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float m_new = fmaxf(m_run, mx);
            // a query whose keys so far are all masked keeps o = 0 and lsum = 0
            const float m_eff = (m_new == -INFINITY) ? 0.0f : m_new;
            if (c0 > 0) {
                const float alpha = (m_run == -INFINITY)
                                        ? 0.0f
                                        : __builtin_amdgcn_exp2f((m_run - m_eff) * kLog2e);
                lsum *= alpha;
#pragma unroll
                for (int i = 0; i < 16; ++i) o[i] *= alpha;
            }
            m_run = m_new;
            const float m2 = m_eff * kLog2e;
            // ---- pass 2: probabilities (unnormalised), row sum, O^T += V^T P^T
#pragma unroll
            for (int kc = 0; kc < KC; ++kc) {
                const int kt = c0 + kc;
                if (__builtin_amdgcn_readfirstlane(kbits[kt]) == 0) continue;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kc][i], kLog2e, -m2));
                    s[kc][i] = p;
                    lsum += p;
                }
                const typename Tr<T>::K32 pb = Tr<T>::pack(s[kc]);
                typename Tr<T>::K32 va;
                if (vrow < D) va = load_k32<T>(&vt_lds[vrow * VSTR + kt * 32], h2);
                else va = zero_k32<T>();
                Tr<T>::mma_k32(o, va, pb);
            }
        }
        lsum += __shfl_xor(lsum, 32);
        const float m_use = m_run;

        // ---- epilogue: normalise, gate, store O and lse
        if (qvalid) {
            const float inv = lsum > 0.0f ? 1.0f / lsum : 0.0f;
            const int64_t tok = base + (int64_t)qi * a.stok;
            const E *G = a.g ? (const E *)a.g + tok : nullptr;
            E *O = (E *)a.out + tok;
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int c0 = 16 * half + 8 * h2;  // channels of regs 8*half .. 8*half+7
                if (c0 >= D) continue;
                float val[8];
#pragma unroll
                for (int s8 = 0; s8 < 8; ++s8) val[s8] = o[8 * half + s8] * inv;
                if (G) {
#pragma unroll
                    for (int s8 = 0; s8 < 8; ++s8) {
                        const float gv = Tr<T>::to_f(G[c0 + s8]);
                        val[s8] = val[s8] / (1.0f + __builtin_amdgcn_exp2f(-gv * kLog2e));
                    }
                }
                if constexpr (sizeof(E) == 2) {
                    uint4 w;
                    w.x = (uint32_t)f2bf(val[0]) | ((uint32_t)f2bf(val[1]) << 16);
                    w.y = (uint32_t)f2bf(val[2]) | ((uint32_t)f2bf(val[3]) << 16);
                    w.z = (uint32_t)f2bf(val[4]) | ((uint32_t)f2bf(val[5]) << 16);
                    w.w = (uint32_t)f2bf(val[6]) | ((uint32_t)f2bf(val[7]) << 16);
                    *reinterpret_cast<uint4 *>(O + c0) = w;
                } else {
                    *reinterpret_cast<float4 *>(O + c0) = make_float4(val[0], val[1], val[2], val[3]);
                    *reinterpret_cast<float4 *>(O + c0 + 4) = make_float4(val[4], val[5], val[6], val[7]);
                }
            }
            if (h2 == 0)
                a.lse[(r * a.H + hh) * a.L + qi] = lsum > 0.0f ? m_use + logf(lsum) : -INFINITY;
        }
    }
}

template <typename T, int D, int NKT>
hipError_t launch_t(const Problem &p, const FwdPtrs &x, hipStream_t s) {
    FwdArgs a;
    a.q = x.q; a.k = x.k; a.v = x.v; a.g = x.g; a.bias = x.bias; a.mask = x.mask;
    a.out = x.out; a.lse = x.lse;
    a.L = p.L; a.rpb = p.rpb; a.srow = p.srow; a.stok = p.stok; a.H = p.H;
    a.scale = 1.0f / sqrtf((float)D);
    constexpr int NW = NKT < 4 ? NKT : 4;
    const int64_t blocks = p.N * p.H;
    hipLaunchKernelGGL((fwd_kernel<T, D, NKT>), dim3((unsigned)blocks), dim3(NW * 64), 0, s, a);
    return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_d(const Problem &p, const FwdPtrs &x, hipStream_t s) {
    const int64_t nkt = (p.L + 31) / 32;
    if (nkt <= 1) return launch_t<T, D, 1>(p, x, s);
    if (nkt <= 2) return launch_t<T, D, 2>(p, x, s);
    if (nkt <= 4) return launch_t<T, D, 4>(p, x, s);
    return launch_t<T, D, 8>(p, x, s);
}

template <typename T>
hipError_t launch_dt(const Problem &p, const FwdPtrs &x, hipStream_t s) {
    switch (p.D) {
        case 8: return launch_d<T, 8>(p, x, s);
        case 16: return launch_d<T, 16>(p, x, s);
        default: return launch_d<T, 32>(p, x, s);
    }
}

}  // namespace

hipError_t launch_fwd(const Problem &p, const FwdPtrs &x, hipStream_t s) {
    if (p.dtype == 1) return launch_dt<bf16_t>(p, x, s);
    return launch_dt<float>(p, x, s);
}

}  // namespace evo
