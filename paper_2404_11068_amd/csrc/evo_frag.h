// evo_frag.h -- gfx950 MFMA fragment helpers shared by the attention kernels.
//
// Every tile product in the kernels is a 32x32 output tile produced by one of
//   v_mfma_f32_32x32x16_bf16   (bf16 inputs, k = 16)
//   v_mfma_f32_32x32x8_bf16    (bf16 inputs, k = 8; head_dim 8)
//   v_mfma_f32_32x32x2_f32     (fp32 inputs, k = 2)
// Lane layout (wave64, lane l, half h = l / 32, col n = l % 32):
//   A operand: row m = l % 32, k-slots h*kpl .. h*kpl + kpl - 1
//   B operand: col n = l % 32, same k-slots
//   D (16 fp32 regs): reg i holds D[rho(i, h)][n],  rho(i, h) = 8*(i/4) + 4*h + i%4
//
// Two index maps make the D layout directly reusable as an MFMA operand:
//   * the rows of an A operand are loaded permuted by sig(m) (bits 2 and 3 of
//     m swapped), so reg i of the product holds row krow(i, h) of the tile:
//         krow(i, h) = 16*(i/8) + 8*h + i%8
//   * a contraction over a 32-row block therefore uses, per lane half h, the
//     rows {8h + s, 16 + 8h + s : s = 0..7} in register order -- the "k32"
//     fragment below -- for both bf16 (2 MFMAs of k=16) and fp32 (16 MFMAs
//     of k=2).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace evo {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef short short4v __attribute__((ext_vector_type(4)));

struct bf16_t { uint16_t bits; };   // storage type of the bf16 path

// ---------------------------------------------------------------------------
// Buffer-resource memory access.  A resource covers [base, base + bytes);
// a load at an offset past the end reads zeros and a store there is dropped
// by the hardware, so out-of-range lanes need no branch: every vector-memory
// instruction is issued unconditionally, which keeps the compiler's in-order
// load counters exact across software-pipelined loads.
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
// Note: __builtin_bit_cast applied to a vector COMPONENT (x.y, x[1]) reads
// component 0 with this compiler; bit-cast whole vectors, then take
// components of the result.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr uint32_t kOOB = 0x80000000u;  // past every resource (sizes stay below 2^31)

__device__ __forceinline__ rsrc_t make_buf(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ u32x4 bload16(rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}
__device__ __forceinline__ u32x2 bload8(rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
}
__device__ __forceinline__ uint32_t bload4(rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}
__device__ __forceinline__ uint16_t bload2(rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
}
__device__ __forceinline__ uint8_t bload1(rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b8(r, off, 0, 0);
}
__device__ __forceinline__ void bstore16(u32x4 v, rsrc_t r, uint32_t off) {
    __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, 0);
}
__device__ __forceinline__ void bstore4(uint32_t v, rsrc_t r, uint32_t off) {
    __builtin_amdgcn_raw_buffer_store_b32(v, r, off, 0, 0);
}

__device__ __forceinline__ int sig(int m) { return (m & ~0xC) | ((m & 4) << 1) | ((m & 8) >> 1); }
__device__ __forceinline__ int krow(int i, int h) { return 16 * (i >> 3) + 8 * h + (i & 7); }

__device__ __forceinline__ float bf2f(uint16_t u) { return __builtin_bit_cast(float, (uint32_t)u << 16); }
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

// ---------------------------------------------------------------------------
// per-dtype traits: element type, 16-byte vector width, MFMA wrappers
template <typename T> struct Tr;

template <> struct Tr<float> {
    using elem = float;
    static constexpr int VEC = 4;  // elements per 16 bytes
    __device__ __forceinline__ static float to_f(float x) { return x; }
    __device__ __forceinline__ static float from_f(float x) { return x; }
    // k32 fragment: 16 floats, MFMA u contracts rows {krow(u,0), krow(u,1)}
    struct K32 { float v[16]; };
    __device__ __forceinline__ static void mma_k32(f32x16 &acc, const K32 &a, const K32 &b) {
#pragma unroll
        for (int u = 0; u < 16; ++u) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.v[u], b.v[u], acc, 0, 0, 0);
    }
    __device__ __forceinline__ static K32 pack(const f32x16 &x) {
        K32 r;
#pragma unroll
        for (int i = 0; i < 16; ++i) r.v[i] = x[i];
        return r;
    }
};

template <> struct Tr<bf16_t> {
    using elem = uint16_t;
    static constexpr int VEC = 8;
    __device__ __forceinline__ static float to_f(uint16_t x) { return bf2f(x); }
    __device__ __forceinline__ static uint16_t from_f(float x) { return f2bf(x); }
    struct K32 { bf16x8 v[2]; };
    __device__ __forceinline__ static void mma_k32(f32x16 &acc, const K32 &a, const K32 &b) {
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a.v[0], b.v[0], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a.v[1], b.v[1], acc, 0, 0, 0);
    }
    __device__ __forceinline__ static K32 pack(const f32x16 &x) {
        K32 r;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            r.v[0][s] = (__bf16)x[s];
            r.v[1][s] = (__bf16)x[8 + s];
        }
        return r;
    }
};

// Load a k32 fragment from a row of 32 consecutive elements (rows of the
// contraction) -- the lane takes elements {8h+s, 16+8h+s}.
template <typename T>
__device__ __forceinline__ typename Tr<T>::K32 load_k32(const typename Tr<T>::elem *row32, int h) {
    typename Tr<T>::K32 f;
    if constexpr (sizeof(typename Tr<T>::elem) == 2) {
        f.v[0] = *reinterpret_cast<const bf16x8 *>(row32 + 8 * h);
        f.v[1] = *reinterpret_cast<const bf16x8 *>(row32 + 16 + 8 * h);
    } else {
        const float4 *p0 = reinterpret_cast<const float4 *>(row32 + 8 * h);
        const float4 *p1 = reinterpret_cast<const float4 *>(row32 + 16 + 8 * h);
        float4 a = p0[0], b = p0[1], c = p1[0], d = p1[1];
        f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
        f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
        f.v[8] = c.x; f.v[9] = c.y; f.v[10] = c.z; f.v[11] = c.w;
        f.v[12] = d.x; f.v[13] = d.y; f.v[14] = d.z; f.v[15] = d.w;
    }
    return f;
}

template <typename T>
__device__ __forceinline__ typename Tr<T>::K32 zero_k32() {
    typename Tr<T>::K32 f;
    if constexpr (sizeof(typename Tr<T>::elem) == 2) {
#pragma unroll
        for (int s = 0; s < 8; ++s) { f.v[0][s] = (__bf16)0.0f; f.v[1][s] = (__bf16)0.0f; }
    } else {
#pragma unroll
        for (int u = 0; u < 16; ++u) f.v[u] = 0.0f;
    }
    return f;
}

// ---------------------------------------------------------------------------
// Channel-contraction fragments (QK^T and dA V^T): contraction over the D
// channels of a token.  The channel order inside the contraction is free, so
// each dtype uses the order that makes the lane's channels contiguous.
template <typename T, int D> struct ChFrag;

// fp32: D/2 MFMAs of k=2; lane half h holds channels h*D/2 + u, u < D/2
template <int D> struct ChFrag<float, D> {
    float v[D / 2];
    // tok = byte offset of the token's D channels in resource r
    __device__ __forceinline__ void load(rsrc_t r, uint32_t tok, int h) {
#pragma unroll
        for (int u = 0; u < D / 2; u += 4) {
            const f32x4 x = __builtin_bit_cast(f32x4, bload16(r, tok + (uint32_t)(h * (D / 2) + u) * 4u));
            v[u] = x.x; v[u + 1] = x.y; v[u + 2] = x.z; v[u + 3] = x.w;
        }
    }
    __device__ __forceinline__ void load(const float *tok, int h) {
#pragma unroll
        for (int u = 0; u < D / 2; u += 4) {
            float4 x = *reinterpret_cast<const float4 *>(tok + h * (D / 2) + u);
            v[u] = x.x; v[u + 1] = x.y; v[u + 2] = x.z; v[u + 3] = x.w;
        }
    }
    __device__ __forceinline__ void zero() {
#pragma unroll
        for (int u = 0; u < D / 2; ++u) v[u] = 0.0f;
    }
    __device__ __forceinline__ static void mma(f32x16 &acc, const ChFrag &a, const ChFrag &b) {
#pragma unroll
        for (int u = 0; u < D / 2; ++u) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.v[u], b.v[u], acc, 0, 0, 0);
    }
};

// bf16, D multiple of 16: D/16 MFMAs of k=16; lane half h holds channels 16kk + 8h + s
template <int D> struct ChFrag<bf16_t, D> {
    static_assert(D % 16 == 0, "bf16 head_dim 16/32 use k=16 MFMAs");
    bf16x8 v[D / 16];
    __device__ __forceinline__ void load(rsrc_t r, uint32_t tok, int h) {
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk)
            v[kk] = __builtin_bit_cast(bf16x8, bload16(r, tok + (uint32_t)(16 * kk + 8 * h) * 2u));
    }
    __device__ __forceinline__ void load(const uint16_t *tok, int h) {
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) v[kk] = *reinterpret_cast<const bf16x8 *>(tok + 16 * kk + 8 * h);
    }
    __device__ __forceinline__ void zero() {
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk)
#pragma unroll
            for (int s = 0; s < 8; ++s) v[kk][s] = (__bf16)0.0f;
    }
    __device__ __forceinline__ static void mma(f32x16 &acc, const ChFrag &a, const ChFrag &b) {
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk)
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a.v[kk], b.v[kk], acc, 0, 0, 0);
    }
};

// bf16, D = 8: one MFMA of k=8; lane half h holds channels 4h + s, s < 4
template <> struct ChFrag<bf16_t, 8> {
    short4v v;
    __device__ __forceinline__ void load(rsrc_t r, uint32_t tok, int h) {
        v = __builtin_bit_cast(short4v, bload8(r, tok + (uint32_t)(4 * h) * 2u));
    }
    __device__ __forceinline__ void load(const uint16_t *tok, int h) {
        v = *reinterpret_cast<const short4v *>(tok + 4 * h);
    }
    __device__ __forceinline__ void zero() { v = short4v{0, 0, 0, 0}; }
    __device__ __forceinline__ static void mma(f32x16 &acc, const ChFrag &a, const ChFrag &b) {
        acc = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(a.v, b.v, acc, 0, 0, 0);
    }
};

// bf16, D = 8 on the k=16 instruction, which on gfx950 issues in about 80% of
// the time of the k=8 one: lane half 0 holds the 8 channels, lane half 1
// k-slots 8..15, which carry one extra rank-1 term of the product.  An LDS row
// of 16 elements holds the 8 channels and then the row's slots 8..15; a token
// loaded from memory gets `slot8` in slot 8 and zeros after it.
struct Frag8K16 {
    bf16x8 v;
    __device__ __forceinline__ void load(rsrc_t r, uint32_t tok, int h, short slot8) {
        u32x4 x = bload16(r, h == 0 ? tok : kOOB);
        x.x = h == 0 ? x.x : (uint32_t)(uint16_t)slot8;
        v = __builtin_bit_cast(bf16x8, x);
    }
    // as above with slots 8..11 of lane half 1 given as two words (low half first)
    __device__ __forceinline__ void load(rsrc_t r, uint32_t tok, int h, uint32_t w0, uint32_t w1) {
        u32x4 x = bload16(r, h == 0 ? tok : kOOB);
        x.x = h == 0 ? x.x : w0;
        x.y = h == 0 ? x.y : w1;
        v = __builtin_bit_cast(bf16x8, x);
    }
    // slot 8 (lane half 1) set after the load
    __device__ __forceinline__ void set_slot8(int h, short s8) {
        u32x4 x = __builtin_bit_cast(u32x4, v);
        x.x = h == 0 ? x.x : (uint32_t)(uint16_t)s8;
        v = __builtin_bit_cast(bf16x8, x);
    }
    __device__ __forceinline__ void load(const uint16_t *row, int h) {
        v = *reinterpret_cast<const bf16x8 *>(row + 8 * h);
    }
    __device__ __forceinline__ static void mma(f32x16 &acc, const Frag8K16 &a, const Frag8K16 &b) {
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a.v, b.v, acc, 0, 0, 0);
    }
};

// operand fragment of a product over the head channels: bf16 at D = 8 takes
// the k=16 form above
template <typename T, int D> struct QKFragSel { using type = ChFrag<T, D>; };
template <> struct QKFragSel<bf16_t, 8> { using type = Frag8K16; };

// ---------------------------------------------------------------------------
// k32 A operand of a contraction over 32 rows of a row-major bf16 LDS tile X
// (X[row][col], `stride` elements per row), where the operand's row m is
// column sig(m) of X and its k-slots are rows kbase + {8h+s, 16+8h+s}:
//     A[m][k] = X[kbase + k][sig(m)]      (a transposed read of X)
// Built from ds_read_b64_tr_b16: within each 16-lane group, output lane j
// element e receives element j%4 of the 8-byte chunk addressed by source lane
// 4e + j/4 of that group.  Source lane i of group G therefore addresses
// row kbase + 16t + 8(G/2) + 4u + i/4, columns c0(i) .. c0(i)+3 with
// c0 = 16(G%2) + 4*sig2(i%4) (sig2 swaps the two bits), for MFMA t and half u.
// Columns >= ncols (head_dim) come out as zero.
typedef short short4tr __attribute__((ext_vector_type(4)));
typedef short short8tr __attribute__((ext_vector_type(8)));

// With zero_cols false the lanes whose operand row is a channel >= ncols keep
// what the read gave them (finite data of the tile): enough wherever those
// rows only feed output rows that are never stored.
__device__ __forceinline__ Tr<bf16_t>::K32 load_k32_tr(const uint16_t *X, int stride, int kbase, int ncols,
                                                      int lane, bool ones_row = false, bool zero_cols = true) {
    const int G = lane >> 4, i = lane & 15;
    const int q = i & 3;
    int c0 = 16 * (G & 1) + 4 * (((q & 1) << 1) | (q >> 1));
    const bool col_ok = c0 < ncols;
    if (!col_ok) c0 = 0;  // keep the address inside the tile; the lanes fed by it are zeroed below
    const int rbase = kbase + 8 * (G >> 1) + (i >> 2);
    Tr<bf16_t>::K32 f;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const uint16_t *src = X + (rbase + 16 * t) * stride + c0;
        const short4tr lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4tr *)(src));
        const short4tr hi =
            __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4tr *)(src + 4 * stride));
        // whole-vector concatenation: element-wise __bf16 insertion of these
        // results was miscompiled (only the first dword of each read survived)
        const short8tr both = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        f.v[t] = __builtin_bit_cast(bf16x8, both);
    }
    // the operand row of this lane is channel sig(lane % 32); with ones_row,
    // channel ncols (< 32) is all ones, so the product also yields column sums
    const int ch = sig(lane & 31);
    if (zero_cols && ch >= ncols) {
        const short v = (ones_row && ch == ncols) ? (short)0x3F80 : (short)0;
        const short8tr w = {v, v, v, v, v, v, v, v};
        f.v[0] = __builtin_bit_cast(bf16x8, w);
        f.v[1] = __builtin_bit_cast(bf16x8, w);
    }
    return f;
}

// ---------------------------------------------------------------------------
// Swizzled LDS tile of bf16 rows of 32 channels (64 bytes, no padding): the
// 16-byte chunk k (channels 8k..8k+7) of row t sits at chunk k ^ ((t >> 2) & 3).
// With 64 four-byte banks, 16 lanes reading one chunk of 16 consecutive rows,
// 16 lanes writing the four chunks of four consecutive rows, and the
// transposing read below (four consecutive rows, all chunks, per 32 lanes)
// all touch each bank once.  A padded 40-element stride left two-way
// conflicts on the row-major writes and the transposing reads.
__device__ __forceinline__ int sw32(int row, int chunk) { return row * 32 + ((chunk ^ ((row >> 2) & 3)) << 3); }

// ChFrag<bf16_t, 32> of `row` from a swizzled tile: channels 16kk + 8h + s
__device__ __forceinline__ void load_sw32(ChFrag<bf16_t, 32> &f, const uint16_t *tile, int row, int h) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) f.v[kk] = *reinterpret_cast<const bf16x8 *>(tile + sw32(row, 2 * kk + h));
}

// load_k32_tr(X, 32, kbase, 32, lane) for a swizzled tile: each lane's
// 8-byte piece lies inside one chunk, so only the chunk index moves
__device__ __forceinline__ Tr<bf16_t>::K32 load_k32_tr_sw32(const uint16_t *X, int kbase, int lane) {
    const int G = lane >> 4, i = lane & 15;
    const int q = i & 3;
    const int c0 = 16 * (G & 1) + 4 * (((q & 1) << 1) | (q >> 1));
    const int rbase = kbase + 8 * (G >> 1) + (i >> 2);
    Tr<bf16_t>::K32 f;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const int r0 = rbase + 16 * t, r1 = r0 + 4;
        const uint16_t *s0 = X + sw32(r0, c0 >> 3) + (c0 & 7);
        const uint16_t *s1 = X + sw32(r1, c0 >> 3) + (c0 & 7);
        const short4tr lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4tr *)(s0));
        const short4tr hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4tr *)(s1));
        const short8tr both = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        f.v[t] = __builtin_bit_cast(bf16x8, both);
    }
    return f;
}

// ---------------------------------------------------------------------------
// A 32 x 32 block of a bf16 pair-bias plane [query][key] (row length L, a
// multiple of 8 so that every 16-byte group lies inside one row), handed to
// the lanes that own keys.
//
// bias_block_load: lane l reads the 16-byte chunks l and l + 64 of the block
// of (query tile qt, key tile kt) as it lies in memory (row = chunk / 4 =
// query, 8 keys per chunk).  Rows past L read zeros.
__device__ __forceinline__ void bias_block_load(rsrc_t rb, int L, int qt, int kt, int lane, u32x4 (&raw)[2]) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int r = (lane >> 2) + 16 * j, cc = lane & 3;
        const int qi = qt * 32 + r;
        raw[j] = bload16(rb, qi < L ? (uint32_t)(qi * L + kt * 32 + 8 * cc) * 2u : kOOB);
    }
}

// bias_block_transpose_raw: the block through a wave's own 32 x 32 LDS tile
// (no barrier: a wave's LDS accesses complete in order), stored with column c
// holding key sig(c) and read back with the transposing read, which hands
// lane n the column sig(n), i.e. key n, at the query rows krow(i, h) of
// register i (packed bf16 in the k32 order) -- the logit layout of a tile
// whose lanes own keys.
__device__ __forceinline__ Tr<bf16_t>::K32 bias_block_transpose_raw(uint16_t *tile, const u32x4 (&raw)[2],
                                                                    int lane) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int r = (lane >> 2) + 16 * j, cc = lane & 3;
        // keys 8cc + 4b + e (e < 4) go to column sig(8cc + 4b + e) = 16(cc/2) + 8b + 4(cc%2) + e
        const int c0 = 16 * (cc >> 1) + 4 * (cc & 1);
        const u32x2 lo = {raw[j].x, raw[j].y}, hi = {raw[j].z, raw[j].w};
        *reinterpret_cast<u32x2 *>(&tile[r * 32 + c0]) = lo;
        *reinterpret_cast<u32x2 *>(&tile[r * 32 + c0 + 8]) = hi;
    }
    return load_k32_tr(tile, 32, 0, 32, lane);
}

// ---------------------------------------------------------------------------
// The pair bias of (query tile qt, key tile kt) as the A operand of a k32
// product: lane m takes the bias row of query qt*32 + sig(m) (the permuted
// rows of the Q operand of S = Q K^T), k-slots = keys kt*32 + {8h+s, 16+8h+s},
// as it lies in memory.  Times sqrt(d) on an identity B operand it adds
// sqrt(d) * bias to the logit tile whose lanes own keys.  BV: rows of whole
// 16-byte groups (two loads per lane); otherwise one element per load.  Rows
// and keys past L read zeros.
template <bool BV>
__device__ __forceinline__ Tr<bf16_t>::K32 bias_rows_k32(rsrc_t rb, int L, int qt, int kt, int lane) {
    const int m = lane & 31, h = lane >> 5;
    const int qi = qt * 32 + sig(m);
    const int k0 = kt * 32 + 8 * h;
    Tr<bf16_t>::K32 f;
    if constexpr (BV) {
        f.v[0] = __builtin_bit_cast(bf16x8, bload16(rb, qi < L ? (uint32_t)(qi * L + k0) * 2u : kOOB));
        f.v[1] = __builtin_bit_cast(bf16x8, bload16(rb, qi < L ? (uint32_t)(qi * L + k0 + 16) * 2u : kOOB));
    } else {
        short8tr w[2];
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int kj = k0 + 16 * t + e;
                w[t][e] = (short)bload2(rb, (qi < L && kj < L) ? (uint32_t)(qi * L + kj) * 2u : kOOB);
            }
        f.v[0] = __builtin_bit_cast(bf16x8, w[0]);
        f.v[1] = __builtin_bit_cast(bf16x8, w[1]);
    }
    return f;
}

// bias_rows_k32<true> with the byte offset of the lane's first group given
// (query row * L + first key) * 2: tiles further down add a constant to it,
// and rows past L land past the end of the resource (zeros).
__device__ __forceinline__ Tr<bf16_t>::K32 bias_rows_k32_at(rsrc_t rb, uint32_t off) {
    Tr<bf16_t>::K32 f;
    f.v[0] = __builtin_bit_cast(bf16x8, bload16(rb, off));
    f.v[1] = __builtin_bit_cast(bf16x8, bload16(rb, off + 32u));
    return f;
}

// An opaque copy of a per-lane value: the compiler cannot see through it, so
// what is computed from the copy stays inside the loop that makes the copy.
// Used where hoisting loop-invariant addresses (one per unrolled step) out of
// a loop would hold more registers than the loop can spare: spilled
// addresses come back through scratch loads, and waiting for those waits for
// every memory operation in flight.
__device__ __forceinline__ uint32_t opaque_u32(uint32_t x) {
    asm volatile("" : "+v"(x));
    return x;
}

// ---------------------------------------------------------------------------
// Constant B operand "c times the identity" for the k32 contraction:
// B[k][n] = c where k == n.  With an A operand holding X[m][k] (k = key of
// the tile, rows in any order), the product adds c * X[m][n] to the tile --
// a [query][key] block read along keys lands in a logit tile whose lanes own
// keys.
__device__ __forceinline__ Tr<bf16_t>::K32 eye_k32(float c, int lane) {
    const int n = lane & 31, h = lane >> 5;
    Tr<bf16_t>::K32 f;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int s = 0; s < 8; ++s) f.v[t][s] = (__bf16)((16 * t + 8 * h + s == n) ? c : 0.0f);
    return f;
}

// sqrt(d) as a sum of two bf16 values (hi + lo matches sqrt(d) to ~3e-7)
__device__ __forceinline__ void sqrt_split(int d, float &hi, float &lo) {
    const float r = sqrtf((float)d);
    hi = (float)(__bf16)r;
    lo = (float)(__bf16)(r - hi);
}

// ---------------------------------------------------------------------------
// Rank-1 MFMA term: acc[m][n] += a(m) * b(n), where a(m) is the bf16 value
// held by lane m (lane half 0) and b(n) the one held by lane n (lane half 0):
// one k-slot of a 32x32x8 product, the other slots zero.  With a = a large
// negative number on masked key rows (or columns) and b = 1, it masks whole
// key rows of a logit tile on the matrix unit instead of per logit.
constexpr short kBf16One = 0x3F80;     // 1.0
constexpr short kBf16MaskNeg = (short)0xDF80;  // -2^64: exp2 of any logit plus this is 0
__device__ __forceinline__ void mma_rank1(f32x16 &acc, short a, short b, int h) {
    const short4v av = {h == 0 ? a : (short)0, 0, 0, 0};
    const short4v bv = {h == 0 ? b : (short)0, 0, 0, 0};
    acc = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(av, bv, acc, 0, 0, 0);
}

__device__ __forceinline__ f32x16 zero16() {
    f32x16 z;
#pragma unroll
    for (int i = 0; i < 16; ++i) z[i] = 0.0f;
    return z;
}

// XCD-aware unit index: consecutive units land on the same XCD (workgroups
// are dispatched round-robin over the 8 XCDs), so the heads of one row share
// that XCD's L2.
__device__ __forceinline__ int64_t xcd_unit(int64_t b, int64_t nb) {
    if (nb % 8 != 0) return b;
    return (b % 8) * (nb / 8) + b / 8;
}

}  // namespace evo
