// evo_ln.hip -- LayerNorm forward and backward kernels, gfx950.
//
// ScaleFold, Section 3.3, "LayerNormalization": AlphaFold normalises rows of
// only 64-256 channels, too short for one workgroup per row to keep the GPU
// busy.  The paper's kernel (a) lets a workgroup handle many rows, (b) gets
// the statistics in one pass over the data, and (c) reduces the weight and
// bias gradients in two steps without atomics (per-block partial sums into a
// buffer, then a per-column sum of that buffer).  The same three points
// shape the kernels here, laid out for wave64 and 16-byte buffer loads:
//
//   * a row of C channels is read by LPR = min(64, C / VEC) lanes, VEC
//     elements (16 bytes) per lane and load, so one wave holds 64 / LPR rows
//     per slot and U slots per pass: every lane has U * NV 16-byte loads in
//     flight before it does any arithmetic.
//   * the row stays in registers after its single read from HBM; the mean is
//     reduced first (of the row minus its first element) and the variance is
//     then reduced from the centred values held in registers.  The paper's
//     single pass of sum and sum of squares would cancel catastrophically for
//     rows whose mean is large against their spread; shifting and centring
//     in registers costs no extra memory traffic.
//   * the backward keeps per-lane column partials of dweight and dbias in
//     registers over all the rows a workgroup visits, folds them across lanes
//     and waves once at the end, and writes one partial row per workgroup; a
//     second kernel sums those rows column by column in a fixed order.
//
// Tails need no branches: each wave addresses its rows through a buffer
// resource that ends at the last row, so loads past it return zeros and
// stores past it are dropped.
#include <stdlib.h>

#include "evo_frag.h"
#include "evo_kernels.h"

namespace evo {
namespace {

constexpr int kLnWaves = 4;     // waves per workgroup

template <typename T, int C_>
struct LnGeom {
    static constexpr int ES = sizeof(T);
    static constexpr int C = C_;
    static constexpr int VEC = 16 / ES;            // elements per 16-byte vector
    static constexpr int NVEC = C_ / VEC;          // vectors per row
    static constexpr int LPR = NVEC < 64 ? NVEC : 64;  // lanes per row
    static constexpr int NV = NVEC / LPR;          // vectors per lane and row
    static constexpr int RPW = 64 / LPR;           // rows per wave slot
    static constexpr int U = NV >= 4 ? 1 : 4 / NV; // slots per pass
    static constexpr int ROWS = RPW * U;           // rows per wave pass
    static_assert(C_ % VEC == 0 && NVEC % LPR == 0, "unsupported row length");
};

// 16 bytes of x as VEC floats
__device__ __forceinline__ void unpack(const u32x4 &raw, float (&f)[8], bf16_t) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        f[2 * i] = __uint_as_float(raw[i] << 16);
        f[2 * i + 1] = __uint_as_float(raw[i] & 0xffff0000u);
    }
}
__device__ __forceinline__ void unpack(const u32x4 &raw, float (&f)[4], float) {
    const f32x4 v = __builtin_bit_cast(f32x4, raw);
#pragma unroll
    for (int i = 0; i < 4; ++i) f[i] = v[i];
}
__device__ __forceinline__ u32x4 pack(const float (&f)[8], bf16_t) {
    bf16x8 b;
#pragma unroll
    for (int i = 0; i < 8; ++i) b[i] = (__bf16)f[i];
    return __builtin_bit_cast(u32x4, b);
}
__device__ __forceinline__ u32x4 pack(const float (&f)[4], float) {
    f32x4 v = {f[0], f[1], f[2], f[3]};
    return __builtin_bit_cast(u32x4, v);
}

// v from another lane of the same 16-lane row, chosen by a DPP control word
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

// Sum over the LPR lanes that share a row (groups of LPR consecutive lanes),
// left in every lane of the group.  Within a 16-lane row the partners come
// through DPP (swap neighbours, swap pairs, mirror each half-row, mirror the
// row: after each step every lane holds the sum of a group twice as large);
// only the 32- and 64-lane steps cross rows through ds_bpermute.
template <int LPR>
__device__ __forceinline__ float row_sum(float v) {
    if constexpr (LPR >= 2) v += dpp<0xB1>(v);   // quad_perm [1,0,3,2]
    if constexpr (LPR >= 4) v += dpp<0x4E>(v);   // quad_perm [2,3,0,1]
    if constexpr (LPR >= 8) v += dpp<0x141>(v);  // row_half_mirror
    if constexpr (LPR >= 16) v += dpp<0x140>(v); // row_mirror
    if constexpr (LPR >= 32) v += __shfl_xor(v, 16, 64);
    if constexpr (LPR >= 64) v += __shfl_xor(v, 32, 64);
    return v;
}

// byte offset of the 16-byte vector v of lane li in a row
template <typename G>
__device__ __forceinline__ uint32_t col_byte(int v, int li) {
    return (uint32_t)((v * G::LPR + li) * G::VEC * G::ES);
}

// the rows of wave pass `it`: a resource that ends at the last row (a pass
// at or past n_pass gets an empty resource, so its loads read zeros)
template <typename G>
__device__ __forceinline__ rsrc_t pass_buf(const void *base, int64_t it, int64_t R, uint32_t elem_bytes_per_row) {
    const int64_t row0 = it * G::ROWS;
    int64_t n = R - row0;
    n = n < 0 ? 0 : (n < G::ROWS ? n : G::ROWS);
    return make_buf((const char *)base + (n > 0 ? row0 * elem_bytes_per_row : 0), (uint32_t)n * elem_bytes_per_row);
}

template <typename G, int U, int NV>
__device__ __forceinline__ void load_pass(u32x4 (&r)[U][NV], rsrc_t rs_, int rs, int li) {
    constexpr uint32_t rbytes = (uint32_t)G::C * G::ES;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int v = 0; v < NV; ++v) r[u][v] = bload16(rs_, (uint32_t)(u * G::RPW + rs) * rbytes + col_byte<G>(v, li));
}

// Persistent: wave-pass `it` runs from the wave's global index in steps of
// the grid's wave count, with the next pass's loads issued before the
// current pass's arithmetic and stores (two passes in flight per wave).
template <typename T, int C>
__global__ __launch_bounds__(64 * kLnWaves) void ln_fwd_kernel(const void *__restrict__ x,
                                                              const float *__restrict__ w,
                                                              const float *__restrict__ b, void *__restrict__ y,
                                                              float *__restrict__ mean, float *__restrict__ rstd,
                                                              int64_t R, float eps) {
    using G = LnGeom<T, C>;
    constexpr int VEC = G::VEC, NV = G::NV, U = G::U;
    constexpr uint32_t rbytes = (uint32_t)C * G::ES;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform: scalar addressing
    const int li = lane % G::LPR, rs = lane / G::LPR;
    const int64_t n_pass = (R + G::ROWS - 1) / G::ROWS;
    const int64_t stride = (int64_t)gridDim.x * kLnWaves;
    int64_t it = (int64_t)blockIdx.x * kLnWaves + wave;
    if (it >= n_pass) return;  // wave-uniform

    u32x4 cur[U][NV], nxt[U][NV];
    load_pass<G>(cur, pass_buf<G>(x, it, R, rbytes), rs, li);
    const rsrc_t rw = make_buf(w, C * 4), rb = make_buf(b, C * 4);
    float wv[NV][VEC], bv[NV][VEC];
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int q = 0; q < VEC / 4; ++q) {
            const uint32_t off = (uint32_t)(((v * G::LPR + li) * VEC + 4 * q) * 4);
            const f32x4 a = __builtin_bit_cast(f32x4, bload16(rw, off));
            const f32x4 c = __builtin_bit_cast(f32x4, bload16(rb, off));
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                wv[v][4 * q + e] = a[e];
                bv[v][4 * q + e] = c[e];
            }
        }
    constexpr float inv_c = 1.0f / (float)C;

    for (; it < n_pass; it += stride) {
        load_pass<G>(nxt, pass_buf<G>(x, it + stride, R, rbytes), rs, li);
        const rsrc_t ry = pass_buf<G>(y, it, R, rbytes);
        const rsrc_t rm = mean ? pass_buf<G>(mean, it, R, 4u) : make_buf(nullptr, 0u);
        const rsrc_t rr = rstd ? pass_buf<G>(rstd, it, R, 4u) : make_buf(nullptr, 0u);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            float f[NV][VEC];
#pragma unroll
            for (int v = 0; v < NV; ++v) unpack(cur[u][v], f[v], T{});
            // shift by the row's first element before summing: the sums then
            // see differences of nearby values, which stay exact where the
            // row's mean is large against its spread
            const float k0 = __shfl(f[0][0], lane & ~(G::LPR - 1), 64);
            float s = 0.f;
#pragma unroll
            for (int v = 0; v < NV; ++v)
#pragma unroll
                for (int e = 0; e < VEC; ++e) {
                    f[v][e] -= k0;
                    s += f[v][e];
                }
            const float mus = row_sum<G::LPR>(s) * inv_c;  // mean - k0
            const float mu = k0 + mus;
            float ss = 0.f;
#pragma unroll
            for (int v = 0; v < NV; ++v)
#pragma unroll
                for (int e = 0; e < VEC; ++e) {
                    f[v][e] -= mus;
                    ss = fmaf(f[v][e], f[v][e], ss);
                }
            const float r = rsqrtf(row_sum<G::LPR>(ss) * inv_c + eps);
            const uint32_t rowb = (uint32_t)(u * G::RPW + rs) * rbytes;
#pragma unroll
            for (int v = 0; v < NV; ++v) {
                float o[VEC];
#pragma unroll
                for (int e = 0; e < VEC; ++e) o[e] = fmaf(f[v][e] * r, wv[v][e], bv[v][e]);
                bstore16(pack(o, T{}), ry, rowb + col_byte<G>(v, li));
            }
            const uint32_t so = li == 0 ? (uint32_t)(u * G::RPW + rs) * 4u : kOOB;
            bstore4(__float_as_uint(mu), rm, so);
            bstore4(__float_as_uint(r), rr, so);
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int v = 0; v < NV; ++v) cur[u][v] = nxt[u][v];
    }
}

// dx for every row, per-workgroup partial column sums of dy * xhat and dy.
// Persistent and pipelined like the forward.
template <typename T, int C>
__global__ __launch_bounds__(64 * kLnWaves) void ln_bwd_kernel(const void *__restrict__ x,
                                                              const float *__restrict__ w,
                                                              const float *__restrict__ mean,
                                                              const float *__restrict__ rstd,
                                                              const void *__restrict__ dy, void *__restrict__ dx,
                                                              float *__restrict__ part, int64_t R) {
    using G = LnGeom<T, C>;
    constexpr int VEC = G::VEC, NV = G::NV, U = G::U;
    constexpr uint32_t rbytes = (uint32_t)C * G::ES;
    __shared__ float red[kLnWaves][2 * C];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform: scalar addressing
    const int li = lane % G::LPR, rs = lane / G::LPR;
    constexpr float inv_c = 1.0f / (float)C;
    const int64_t n_pass = (R + G::ROWS - 1) / G::ROWS;
    const int64_t stride = (int64_t)gridDim.x * kLnWaves;
    int64_t it = (int64_t)blockIdx.x * kLnWaves + wave;

    u32x4 xc[U][NV], gc[U][NV], xn[U][NV], gn[U][NV];
    float mc[U], rc[U], mn[U], rn[U];
    auto load_stats = [&](float (&m)[U], float (&r)[U], int64_t i) {
        const rsrc_t rm = pass_buf<G>(mean, i, R, 4u), rr = pass_buf<G>(rstd, i, R, 4u);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            m[u] = __uint_as_float(bload4(rm, (uint32_t)(u * G::RPW + rs) * 4u));
            r[u] = __uint_as_float(bload4(rr, (uint32_t)(u * G::RPW + rs) * 4u));
        }
    };
    load_pass<G>(xc, pass_buf<G>(x, it, R, rbytes), rs, li);
    load_pass<G>(gc, pass_buf<G>(dy, it, R, rbytes), rs, li);
    load_stats(mc, rc, it);

    const rsrc_t rw = make_buf(w, C * 4);
    float wv[NV][VEC];
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int q = 0; q < VEC / 4; ++q) {
            const f32x4 a = __builtin_bit_cast(
                f32x4, bload16(rw, (uint32_t)(((v * G::LPR + li) * VEC + 4 * q) * 4)));
#pragma unroll
            for (int e = 0; e < 4; ++e) wv[v][4 * q + e] = a[e];
        }
    float pw[NV][VEC], pb[NV][VEC];
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < VEC; ++e) pw[v][e] = pb[v][e] = 0.f;

    for (; it < n_pass; it += stride) {
        load_pass<G>(xn, pass_buf<G>(x, it + stride, R, rbytes), rs, li);
        load_pass<G>(gn, pass_buf<G>(dy, it + stride, R, rbytes), rs, li);
        load_stats(mn, rn, it + stride);
        const rsrc_t rd = pass_buf<G>(dx, it, R, rbytes);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            float xh[NV][VEC], g[NV][VEC];
            float sg = 0.f, sgx = 0.f;
#pragma unroll
            for (int v = 0; v < NV; ++v) {
                float dyf[VEC];
                unpack(xc[u][v], xh[v], T{});
                unpack(gc[u][v], dyf, T{});
#pragma unroll
                for (int e = 0; e < VEC; ++e) {
                    xh[v][e] = (xh[v][e] - mc[u]) * rc[u];
                    g[v][e] = dyf[e] * wv[v][e];
                    sg += g[v][e];
                    sgx = fmaf(g[v][e], xh[v][e], sgx);
                    pw[v][e] = fmaf(dyf[e], xh[v][e], pw[v][e]);
                    pb[v][e] += dyf[e];
                }
            }
            const float a = row_sum<G::LPR>(sg) * inv_c;
            const float c = row_sum<G::LPR>(sgx) * inv_c;
            const uint32_t rowb = (uint32_t)(u * G::RPW + rs) * rbytes;
#pragma unroll
            for (int v = 0; v < NV; ++v) {
                float o[VEC];
#pragma unroll
                for (int e = 0; e < VEC; ++e) o[e] = rc[u] * (g[v][e] - a - xh[v][e] * c);
                bstore16(pack(o, T{}), rd, rowb + col_byte<G>(v, li));
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            mc[u] = mn[u];
            rc[u] = rn[u];
#pragma unroll
            for (int v = 0; v < NV; ++v) {
                xc[u][v] = xn[u][v];
                gc[u][v] = gn[u][v];
            }
        }
    }

    // fold the lanes that hold the same columns (different row slots), in a
    // fixed butterfly order, then the waves in index order through LDS
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
#pragma unroll
            for (int m = G::LPR; m < 64; m <<= 1) {
                pw[v][e] += __shfl_xor(pw[v][e], m, 64);
                pb[v][e] += __shfl_xor(pb[v][e], m, 64);
            }
        }
    if (rs == 0) {
#pragma unroll
        for (int v = 0; v < NV; ++v)
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                const int col = (v * G::LPR + li) * VEC + e;
                red[wave][col] = pw[v][e];
                red[wave][C + col] = pb[v][e];
            }
    }
    __syncthreads();
    const rsrc_t rp = make_buf(part + (int64_t)blockIdx.x * 2 * C, 2 * C * 4);
    for (int col = threadIdx.x; col < 2 * C; col += 64 * kLnWaves) {
        float s = red[0][col];
#pragma unroll
        for (int k = 1; k < kLnWaves; ++k) s += red[k][col];
        bstore4(__float_as_uint(s), rp, (uint32_t)col * 4u);
    }
}

// dweight[c] = sum_k part[k][c], dbias[c] = sum_k part[k][C + c].  Wave sl
// of a workgroup sums rows k = sl, sl + 16, ... of 64 columns in order, with
// kLnRedBatch loads in flight per lane; the 16 slices are then added in order.
constexpr int kLnRedSlices = 16;
constexpr int kLnRedBatch = 16;

__global__ __launch_bounds__(64 * kLnRedSlices) void ln_param_reduce_kernel(const float *__restrict__ part,
                                                                           int n_part, int C,
                                                                           float *__restrict__ dw,
                                                                           float *__restrict__ db) {
    __shared__ float red[kLnRedSlices][64];
    const int lane = threadIdx.x & 63, sl = threadIdx.x >> 6;
    const int col = blockIdx.x * 64 + lane;  // column of the 2C-wide partial row
    const rsrc_t rp = make_buf(part, (uint32_t)n_part * 2u * (uint32_t)C * 4u);
    const bool live = col < 2 * C;
    float s = 0.f;
    for (int k0 = sl; k0 < n_part; k0 += kLnRedSlices * kLnRedBatch) {
        float v[kLnRedBatch];
#pragma unroll
        for (int j = 0; j < kLnRedBatch; ++j) {
            const int k = k0 + j * kLnRedSlices;
            const uint32_t off = (live && k < n_part) ? ((uint32_t)k * 2u * (uint32_t)C + (uint32_t)col) * 4u : kOOB;
            v[j] = __uint_as_float(bload4(rp, off));
        }
#pragma unroll
        for (int j = 0; j < kLnRedBatch; ++j) s += v[j];
    }
    red[sl][lane] = s;
    __syncthreads();
    if (sl == 0 && live) {
        float t = red[0][lane];
        for (int q = 1; q < kLnRedSlices; ++q) t += red[q][lane];
        if (col < C)
            dw[col] = t;
        else
            db[col - C] = t;
    }
}

// Persistent grid sizes (workgroups of kLnWaves waves): enough waves per CU
// to cover HBM latency with two passes in flight each; the backward's count
// is also its number of partial dweight/dbias rows.
int ln_grid_cap(const char *env, int dflt) {
    const char *e = getenv(env);
    const int v = e ? atoi(e) : 0;
    return v > 0 ? v : dflt;
}
constexpr int kLnFwdWgDefault = 1 << 30;  // one pass per wave
constexpr int kLnBwdWgDefault = 512;

template <typename T, int C>
int64_t ln_passes_wg(int64_t R) {
    using G = LnGeom<T, C>;
    const int64_t rows_wg = (int64_t)G::ROWS * kLnWaves;
    return (R + rows_wg - 1) / rows_wg;
}

template <typename T, int C>
hipError_t ln_fwd_c(const LnProblem &p, const LnPtrs &x, hipStream_t s) {
    static const int cap = ln_grid_cap("EVO_LN_FWD_WGS", kLnFwdWgDefault);
    const int64_t n = ln_passes_wg<T, C>(p.R);
    const int64_t nwg = n < cap ? n : cap;
    hipLaunchKernelGGL((ln_fwd_kernel<T, C>), dim3((unsigned)nwg), dim3(64 * kLnWaves), 0, s, x.x, x.w, x.b,
                       x.y, x.mean, x.rstd, p.R, p.eps);
    return hipGetLastError();
}

template <typename T, int C>
int64_t ln_bwd_wgs(int64_t R) {
    static const int cap = ln_grid_cap("EVO_LN_BWD_WGS", kLnBwdWgDefault);
    const int64_t n = ln_passes_wg<T, C>(R);
    return n < cap ? n : cap;
}

template <typename T, int C>
hipError_t ln_bwd_c(const LnProblem &p, const LnBwdPtrs &x, void *ws, hipStream_t s, Tracer *tr) {
    const int64_t nwg = ln_bwd_wgs<T, C>(p.R);
    float *part = (float *)ws;
    if (tr) tr->mark(s);
    if (nwg > 0) {  // with no rows the reduction below writes zeros
        hipLaunchKernelGGL((ln_bwd_kernel<T, C>), dim3((unsigned)nwg), dim3(64 * kLnWaves), 0, s, x.x, x.w,
                           x.mean, x.rstd, x.dy, x.dx, part, p.R);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (tr) tr->mark(s);
    hipLaunchKernelGGL(ln_param_reduce_kernel, dim3((unsigned)((2 * C + 63) / 64)), dim3(64 * kLnRedSlices), 0,
                       s, part, (int)nwg, C, x.dw, x.db);
    hipError_t e = hipGetLastError();
    if (tr) tr->mark(s);
    return e;
}

template <typename T>
hipError_t ln_fwd_t(const LnProblem &p, const LnPtrs &x, hipStream_t s) {
    switch (p.C) {
        case 32: return ln_fwd_c<T, 32>(p, x, s);
        case 64: return ln_fwd_c<T, 64>(p, x, s);
        case 128: return ln_fwd_c<T, 128>(p, x, s);
        case 256: return ln_fwd_c<T, 256>(p, x, s);
        case 512: return ln_fwd_c<T, 512>(p, x, s);
        case 1024: return ln_fwd_c<T, 1024>(p, x, s);
    }
    return hipErrorInvalidValue;
}

template <typename T>
hipError_t ln_bwd_t(const LnProblem &p, const LnBwdPtrs &x, void *ws, hipStream_t s, Tracer *tr) {
    switch (p.C) {
        case 32: return ln_bwd_c<T, 32>(p, x, ws, s, tr);
        case 64: return ln_bwd_c<T, 64>(p, x, ws, s, tr);
        case 128: return ln_bwd_c<T, 128>(p, x, ws, s, tr);
        case 256: return ln_bwd_c<T, 256>(p, x, ws, s, tr);
        case 512: return ln_bwd_c<T, 512>(p, x, ws, s, tr);
        case 1024: return ln_bwd_c<T, 1024>(p, x, ws, s, tr);
    }
    return hipErrorInvalidValue;
}

template <typename T>
int64_t ln_bwd_wgs_t(const LnProblem &p) {
    switch (p.C) {
        case 32: return ln_bwd_wgs<T, 32>(p.R);
        case 64: return ln_bwd_wgs<T, 64>(p.R);
        case 128: return ln_bwd_wgs<T, 128>(p.R);
        case 256: return ln_bwd_wgs<T, 256>(p.R);
        case 512: return ln_bwd_wgs<T, 512>(p.R);
        case 1024: return ln_bwd_wgs<T, 1024>(p.R);
    }
    return 0;
}

}  // namespace

bool ln_supported_cols(int C) {
    return C == 32 || C == 64 || C == 128 || C == 256 || C == 512 || C == 1024;
}

size_t ln_bwd_workspace(const LnProblem &p) {
    const int64_t nwg = p.dtype == 1 ? ln_bwd_wgs_t<bf16_t>(p) : ln_bwd_wgs_t<float>(p);
    return (size_t)(nwg > 0 ? nwg : 1) * 2 * (size_t)p.C * sizeof(float);
}

hipError_t launch_ln_fwd(const LnProblem &p, const LnPtrs &x, hipStream_t s) {
    return p.dtype == 1 ? ln_fwd_t<bf16_t>(p, x, s) : ln_fwd_t<float>(p, x, s);
}

hipError_t launch_ln_bwd(const LnProblem &p, const LnBwdPtrs &x, void *ws, hipStream_t s, Tracer *tr) {
    return p.dtype == 1 ? ln_bwd_t<bf16_t>(p, x, ws, s, tr) : ln_bwd_t<float>(p, x, ws, s, tr);
}

}  // namespace evo
