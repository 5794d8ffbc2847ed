// evo_fwd.hip -- forward kernel of the gated attention with pair bias, gfx950.
//
// o = sigmoid(g) * softmax(Q K^T / sqrt(d) + bias + mask) V, plus the
// per-query log-sum-exp (ScaleFold Section 3.3, "Multi Head Attention": the
// pair bias enters the logits before the softmax; all of MHA in one kernel).
//
// Work unit = one (row, head).  A workgroup has one wave per 32-query tile
// (seq_len <= 256, so at most 8 waves) and is persistent: it walks a strided
// list of units, and while it computes one unit the global loads of the next
// unit's K, V, Q and key mask are already in flight into registers.  K and V
// sit row-major in LDS; the V^T operand of O^T = V^T P^T comes out of the
// transposing LDS read (ds_read_b64_tr_b16) on the bf16 path.
//
// Logits are produced transposed (S^T = K Q^T): a lane owns one query and
// the keys sit in its registers, so row max and row sum are in-lane
// reductions plus one exchange between the two lane halves, and the
// probabilities in registers are already the B operand of O^T = V^T P^T.
// A wave keeps the logits of 128 keys (4 tiles) in registers at a time,
// takes their max and exponentials in two passes over registers, and
// rescales its running sums between such chunks (once at seq_len 256).
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
    int64_t L, rpb, srow, stok, n_units;
    int H;
    float scale;
};

// 8 consecutive values row[j0 .. j0+7] as fp32 (vector load); caller
// guarantees j0 + 8 <= n and 16-byte alignment
template <typename T>
__device__ __forceinline__ void load8_vec(const typename Tr<T>::elem *row, int j0, float *out8) {
    using E = typename Tr<T>::elem;
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
}

template <typename T>
__device__ __forceinline__ void load8_guarded(const typename Tr<T>::elem *row, int j0, int n, float *out8) {
#pragma unroll
    for (int s = 0; s < 8; ++s) out8[s] = (j0 + s < n) ? Tr<T>::to_f(row[j0 + s]) : 0.0f;
}

// unit index handled by workgroup slot `w` at step `it`: each XCD (blockIdx
// % 8) walks its own contiguous share of the units, so the heads of one row
// are processed at the same time on one XCD and share its L2.
__device__ __forceinline__ int64_t unit_of(int64_t w, int64_t it, int64_t nwg, int64_t n_units) {
    if (nwg % 8 != 0) return w + it * nwg;
    const int64_t per_xcd = nwg / 8, x = w % 8, slot = w / 8;
    const int64_t share = (n_units + 7) / 8;
    const int64_t u = x * share + slot + it * per_xcd;
    return (u < (x + 1) * share && u < n_units) ? u : n_units;  // n_units = past the end
}

template <typename T, int D, int NKT>
__global__ void __launch_bounds__(NKT * 64) fwd_kernel(FwdArgs a) {
    using E = typename Tr<T>::elem;
    using K32 = typename Tr<T>::K32;
    constexpr bool kTr = sizeof(E) == 2;  // bf16: V^T fragments via the transposing LDS read
    constexpr int VEC = Tr<T>::VEC;
    constexpr int CPT = D / VEC;          // 16-byte chunks per token
    constexpr int LP = NKT * 32;
    constexpr int NT = NKT * 64;
    constexpr int KSTR = D + VEC;         // row stride of K / V in LDS (elements)
    constexpr int VSTR = LP + VEC;        // row stride of V^T in LDS (fp32 path)
    constexpr int KC = NKT < 4 ? NKT : 4; // key tiles per register-resident chunk
    constexpr int NPF = (LP * CPT + NT - 1) / NT;  // 16-byte chunks of K (and of V) per thread
    __shared__ __attribute__((aligned(16))) E k_lds[LP * KSTR];
    __shared__ __attribute__((aligned(16))) E v_lds[kTr ? LP * KSTR : D * VSTR];
    __shared__ uint32_t kbits[NKT];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h2 = lane >> 5, n = lane & 31;
    const int L = (int)a.L;
    const int qt = wave;
    const int qi = qt * 32 + n;
    const bool qvalid = qi < L;
    const bool bias_vec = (L % VEC) == 0;
    const int64_t nwg = gridDim.x;

    // ---- prefetch registers for one unit
    uint4 kpf[NPF], vpf[NPF];
    ChFrag<T, D> qf;
    bool mpf = false;
    auto prefetch = [&](int64_t u) {
        const int64_t r = u / a.H;
        const int hh = (int)(u % a.H);
        const int64_t base = r * a.srow + (int64_t)hh * D;
#pragma unroll
        for (int j = 0; j < NPF; ++j) {
            const int idx = tid + j * NT;
            const int t = idx / CPT, c = (idx % CPT) * VEC;
            kpf[j] = make_uint4(0, 0, 0, 0);
            vpf[j] = make_uint4(0, 0, 0, 0);
            if (idx < LP * CPT && t < L) {
                kpf[j] = *reinterpret_cast<const uint4 *>((const E *)a.k + base + (int64_t)t * a.stok + c);
                vpf[j] = *reinterpret_cast<const uint4 *>((const E *)a.v + base + (int64_t)t * a.stok + c);
            }
        }
        if (qvalid) qf.load((const E *)a.q + base + (int64_t)qi * a.stok, h2);
        else qf.zero();
        mpf = tid < L && (!a.mask || a.mask[r * a.L + tid] != 0);
    };

    int64_t u = unit_of(blockIdx.x, 0, nwg, a.n_units);
    if (u < a.n_units) prefetch(u);
    for (int64_t it = 0; u < a.n_units; ++it) {
        const int64_t r = u / a.H;
        const int hh = (int)(u % a.H);
        const int64_t base = r * a.srow + (int64_t)hh * D;

        // ---- move the prefetched unit into LDS
        __syncthreads();  // the previous unit's LDS reads are done
#pragma unroll
        for (int j = 0; j < NPF; ++j) {
            const int idx = tid + j * NT;
            if (idx < LP * CPT) {
                const int t = idx / CPT, c = (idx % CPT) * VEC;
                *reinterpret_cast<uint4 *>(&k_lds[t * KSTR + c]) = kpf[j];
                if constexpr (kTr) {
                    *reinterpret_cast<uint4 *>(&v_lds[t * KSTR + c]) = vpf[j];
                } else {
                    const E *ve = reinterpret_cast<const E *>(&vpf[j]);
#pragma unroll
                    for (int e = 0; e < VEC; ++e) v_lds[(c + e) * VSTR + t] = ve[e];
                }
            }
        }
        {
            const unsigned long long bal = __ballot(mpf);  // NT >= LP: one key per thread
            if (lane == 0) {
                if (2 * wave < NKT) kbits[2 * wave] = (uint32_t)bal;
                if (2 * wave + 1 < NKT) kbits[2 * wave + 1] = (uint32_t)(bal >> 32);
            }
        }
        const ChFrag<T, D> qcur = qf;
        __syncthreads();

        // ---- loads of the next unit go out now and land during the compute
        const int64_t un = unit_of(blockIdx.x, it + 1, nwg, a.n_units);
        if (un < a.n_units) prefetch(un);

        const E *bias_row = nullptr;
        if (a.bias && qvalid) bias_row = (const E *)a.bias + (((r / a.rpb) * a.H + hh) * (int64_t)L + qi) * L;

        float m_run = -INFINITY, lsum = 0.0f;
        f32x16 o = zero16();
        for (int c0 = 0; c0 < NKT; c0 += KC) {
            // ---- pass 1: logits of the chunk and their max
            f32x16 s[KC];
            float mx = -INFINITY;
#pragma unroll
            for (int kc = 0; kc < KC; ++kc) {
                const int kt = c0 + kc;
                const uint32_t kb = __builtin_amdgcn_readfirstlane(kbits[kt]);
                if (kb == 0) continue;
                ChFrag<T, D> kf;
                kf.load(&k_lds[(kt * 32 + sig(n)) * KSTR], h2);
                s[kc] = zero16();
                ChFrag<T, D>::mma(s[kc], kf, qcur);
                float b[16];
                if (bias_row) {
                    if (bias_vec && (kt + 1) * 32 <= L) {  // whole tile in range (uniform)
                        load8_vec<T>(bias_row, kt * 32 + 8 * h2, b);
                        load8_vec<T>(bias_row, kt * 32 + 16 + 8 * h2, b + 8);
                    } else {
                        load8_guarded<T>(bias_row, kt * 32 + 8 * h2, L, b);
                        load8_guarded<T>(bias_row, kt * 32 + 16 + 8 * h2, L, b + 8);
                    }
                } else {
#pragma unroll
                    for (int i = 0; i < 16; ++i) b[i] = 0.0f;
                }
                if (kb == 0xffffffffu) {
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        s[kc][i] = __builtin_fmaf(s[kc][i], a.scale, b[i]);
                        mx = fmaxf(mx, s[kc][i]);
                    }
                } else {
                    const uint32_t kbl = kb >> (8 * h2);
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const float t = __builtin_fmaf(s[kc][i], a.scale, b[i]);
                        s[kc][i] = ((kbl >> (16 * (i >> 3) + (i & 7))) & 1u) ? t : -INFINITY;
                        mx = fmaxf(mx, s[kc][i]);
                    }
                }
            }
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float m_new = fmaxf(m_run, mx);
            // a query whose keys so far are all masked keeps o = 0 and lsum = 0
            const float m_eff = (m_new == -INFINITY) ? 0.0f : m_new;
            if (c0 > 0) {
                const float alpha =
                    (m_run == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f((m_run - m_eff) * kLog2e);
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
                const K32 pb = Tr<T>::pack(s[kc]);
                K32 va;
                if constexpr (kTr) {
                    va = load_k32_tr(v_lds, KSTR, kt * 32, D, lane);
                } else {
                    if (sig(n) < D) va = load_k32<T>(&v_lds[sig(n) * VSTR + kt * 32], h2);
                    else va = zero_k32<T>();
                }
                Tr<T>::mma_k32(o, va, pb);
            }
        }
        lsum += __shfl_xor(lsum, 32);

        // ---- epilogue: normalise, gate, store O and lse
        if (qvalid) {
            const float inv = lsum > 0.0f ? __builtin_amdgcn_rcpf(lsum) : 0.0f;
            const int64_t tok = base + (int64_t)qi * a.stok;
            const E *G = a.g ? (const E *)a.g + tok : nullptr;
            E *O = (E *)a.out + tok;
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int cb = 16 * half + 8 * h2;  // channels of regs 8*half .. 8*half+7
                if (cb >= D) continue;
                float val[8];
#pragma unroll
                for (int s8 = 0; s8 < 8; ++s8) val[s8] = o[8 * half + s8] * inv;
                if (G) {
                    float gv[8];
                    load8_vec<T>(G, cb, gv);
#pragma unroll
                    for (int s8 = 0; s8 < 8; ++s8) val[s8] *= __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-gv[s8] * kLog2e));
                }
                if constexpr (sizeof(E) == 2) {
                    uint4 w;
                    w.x = (uint32_t)f2bf(val[0]) | ((uint32_t)f2bf(val[1]) << 16);
                    w.y = (uint32_t)f2bf(val[2]) | ((uint32_t)f2bf(val[3]) << 16);
                    w.z = (uint32_t)f2bf(val[4]) | ((uint32_t)f2bf(val[5]) << 16);
                    w.w = (uint32_t)f2bf(val[6]) | ((uint32_t)f2bf(val[7]) << 16);
                    *reinterpret_cast<uint4 *>(O + cb) = w;
                } else {
                    *reinterpret_cast<float4 *>(O + cb) = make_float4(val[0], val[1], val[2], val[3]);
                    *reinterpret_cast<float4 *>(O + cb + 4) = make_float4(val[4], val[5], val[6], val[7]);
                }
            }
            if (h2 == 0)
                a.lse[(r * a.H + hh) * a.L + qi] = lsum > 0.0f ? m_run + logf(lsum) : -INFINITY;
        }
        u = un;
    }
}

template <typename T, int D, int NKT>
hipError_t launch_t(const Problem &p, const FwdPtrs &x, hipStream_t s) {
    FwdArgs a;
    a.q = x.q; a.k = x.k; a.v = x.v; a.g = x.g; a.bias = x.bias; a.mask = x.mask;
    a.out = x.out; a.lse = x.lse;
    a.L = p.L; a.rpb = p.rpb; a.srow = p.srow; a.stok = p.stok; a.H = p.H;
    a.n_units = p.N * p.H;
    a.scale = 1.0f / sqrtf((float)D);
    // persistent grid: as many workgroups as fit on the chip at once (queried
    // once per kernel instantiation), never more than units
    static const int per_cu = [] {
        int nb = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, fwd_kernel<T, D, NKT>, NKT * 64, 0) != hipSuccess ||
            nb < 1)
            nb = 1;
        return nb;
    }();
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        cus = 256;
    int64_t nwg = (int64_t)cus * per_cu;
    if (nwg > a.n_units) nwg = a.n_units;
    hipLaunchKernelGGL((fwd_kernel<T, D, NKT>), dim3((unsigned)nwg), dim3(NKT * 64), 0, s, a);
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
