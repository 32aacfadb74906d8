// Device helpers for gfx950: bfloat16 conversion, 16x16x32 MFMA tiles on
// 8-element fragments, Philox4x64-10 and LSTM activations.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lsd {

typedef uint16_t bf16;   // raw bfloat16 bits

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short s16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(bf16 h) { return __uint_as_float((uint32_t)h << 16); }

// float -> bfloat16, round to nearest even (finite inputs)
__device__ __forceinline__ bf16 f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (bf16)(u >> 16);
}

template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<bf16>(bf16 v) { return bf2f(v); }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) { return f2bf(v); }

template <typename T> __device__ __forceinline__ T zero_val() { return (T)0; }

// An MFMA operand fragment: 8 consecutive contraction elements of one row
// (A) or one column (B) held by one lane.  For the 16x16 tile, lane l holds
// row/column l%16 and contraction elements 8*(l/16) .. 8*(l/16)+7 of a
// 32-long contraction chunk.  The contraction order inside a chunk only has
// to agree between A and B, so the fp32 path issues the 4-deep fp32 MFMA
// once per fragment slot.
template <typename T> struct Frag { T v[8]; };

__device__ __forceinline__ void mma_16x16x32(const Frag<bf16>& a, const Frag<bf16>& b, f32x4_t& c) {
    s16x8_t av, bv;
#pragma unroll
    for (int e = 0; e < 8; ++e) { av[e] = (short)a.v[e]; bv[e] = (short)b.v[e]; }
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, av),
                                                __builtin_bit_cast(bf16x8_t, bv), c, 0, 0, 0);
}

__device__ __forceinline__ void mma_16x16x32(const Frag<float>& a, const Frag<float>& b, f32x4_t& c) {
#pragma unroll
    for (int e = 0; e < 8; ++e) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[e], b.v[e], c, 0, 0, 0);
}

// Fragment-major layout of a [rows][cols] matrix whose rows are the M side
// of an MFMA product: 32-column chunks x 16-row tiles x 64 lanes x 8
// elements.  Element (row, col) of a matrix with `mtiles` 16-row tiles sits
// at frag_off(row, col, mtiles); the A fragment of (chunk c, tile mt) is the
// 16 bytes of lane l at frag_lane_off(c, mt, l, mtiles), and a wave reads it
// as one contiguous 1 KB block.  A buffer holds ceil(cols/32)*mtiles*512
// elements.
__device__ __forceinline__ size_t frag_lane_off(int c, int mt, int lane, int mtiles) {
    return (((size_t)c * mtiles + mt) * 64 + lane) << 3;
}
__device__ __forceinline__ size_t frag_off(int row, int col, int mtiles) {
    const int k = col & 31;
    return frag_lane_off(col >> 5, row >> 4, (k >> 3) * 16 + (row & 15), mtiles) + (k & 7);
}

// 8 consecutive elements (16-byte aligned bf16, 32-byte aligned f32)
__device__ __forceinline__ void ld8(const bf16* p, bf16* o) {
    const uint4 v = *(const uint4*)p;
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = (bf16)((w[e >> 1] >> (16 * (e & 1))) & 0xffffu);
}
__device__ __forceinline__ void ld8(const float* p, float* o) {
    const float4 v0 = *(const float4*)p, v1 = *(const float4*)(p + 4);
    o[0] = v0.x; o[1] = v0.y; o[2] = v0.z; o[3] = v0.w;
    o[4] = v1.x; o[5] = v1.y; o[6] = v1.z; o[7] = v1.w;
}

// ---------------------------------------------------------------------------
// Buffer-resource loads (32-bit offsets; reads past the resource return 0)
// and 8-element operand fragments held as packed dwords.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
constexpr int BUF_FLAGS = 0x00020000;             // raw 32-bit buffer resource word 3 (gfx9)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, BUF_FLAGS);
}
// 8 consecutive elements of one operand row as packed dwords
template <typename T> struct Raw8 { static constexpr int NW = 4 * (int)sizeof(T) / 2; uint32_t w[NW]; };

// cache-policy bits of a buffer load: SC1 makes it device-coherent (it reads
// at the device's coherence point, past the per-XCD L2, whatever the caches
// hold), the form of an agent-scope atomic load
constexpr int CPOL_SC1 = 16;

template <typename T, int CPOL = 0>
__device__ __forceinline__ void raw_load(Raw8<T>& f, __amdgpu_buffer_rsrc_t r, uint32_t off) {
#pragma unroll
    for (int q = 0; q < Raw8<T>::NW / 4; ++q) {
        const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, off + 16 * q, 0, CPOL);
#pragma unroll
        for (int e = 0; e < 4; ++e) f.w[4 * q + e] = v[e];
    }
}
// A buffer offset past every resource: the load returns 0 and moves no data.
// Used for A-fragment lanes whose row lies past the batch.
constexpr uint32_t OOB_OFF = 0x80000000u;

// AND masks that zero the elements at index >= B of a fragment whose first
// element sits at index b0
template <typename T>
__device__ __forceinline__ void pad_mask(int b0, int B, uint32_t* m) {
    if (sizeof(T) == 2) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
            m[q] = (b0 + 2 * q < B ? 0x0000ffffu : 0u) | (b0 + 2 * q + 1 < B ? 0xffff0000u : 0u);
    } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) m[q] = b0 + q < B ? 0xffffffffu : 0u;
    }
}
template <typename T>
__device__ __forceinline__ void raw_and(Raw8<T>& f, const uint32_t* m) {
#pragma unroll
    for (int q = 0; q < Raw8<T>::NW; ++q) f.w[q] &= m[q];
}
__device__ __forceinline__ void raw_mma(const Raw8<bf16>& a, const Raw8<bf16>& b, f32x4_t& c) {
    const u32x4_t av = {a.w[0], a.w[1], a.w[2], a.w[3]}, bv = {b.w[0], b.w[1], b.w[2], b.w[3]};
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, av), __builtin_bit_cast(bf16x8_t, bv),
                                                c, 0, 0, 0);
}
__device__ __forceinline__ void raw_mma(const Raw8<float>& a, const Raw8<float>& b, f32x4_t& c) {
#pragma unroll
    for (int e = 0; e < 8; ++e)
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w[e]), __uint_as_float(b.w[e]), c, 0, 0, 0);
}

// column sums of a packed fragment (bias gradient)
template <typename T>
__device__ __forceinline__ void db_add_raw(const Raw8<T>& f, float& acc) {
    if (sizeof(T) == 2) {
#pragma unroll
        for (int q = 0; q < Raw8<T>::NW; ++q) acc += __uint_as_float(f.w[q] << 16) + __uint_as_float(f.w[q] & 0xffff0000u);
    } else {
#pragma unroll
        for (int q = 0; q < Raw8<T>::NW; ++q) acc += __uint_as_float(f.w[q]);
    }
}

// 8 elements from LDS (16-byte aligned)
template <typename T>
__device__ __forceinline__ void raw_lds(Raw8<T>& f, const T* p) {
#pragma unroll
    for (int q = 0; q < Raw8<T>::NW / 4; ++q) {
        const uint4 v = *(const uint4*)((const char*)p + 16 * q);
        f.w[4 * q] = v.x; f.w[4 * q + 1] = v.y; f.w[4 * q + 2] = v.z; f.w[4 * q + 3] = v.w;
    }
}
// Four consecutive 16-bit elements through the transposing LDS read of
// gfx950 (ds_read_b64_tr_b16).  Within each 16-lane group, lane i receives
// element i % 4 of the 8 bytes addressed by lanes 4e + i / 4, e = 0..3, as
// its element e: when lanes 4e..4e+3 address columns 0, 4, 8, 12 of one row
// of a K-major [K][N] tile, lane i receives column i of the four rows e.
typedef short s16x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint2 lds_tr4(const bf16* p) {
    const s16x4_t r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((s16x4_t __attribute__((address_space(3)))*)p);
    return __builtin_bit_cast(uint2, r);
}

// pack an element-wise fragment
__device__ __forceinline__ void raw_from(Raw8<bf16>& f, const Frag<bf16>& x) {
#pragma unroll
    for (int q = 0; q < 4; ++q) f.w[q] = (uint32_t)x.v[2 * q] | ((uint32_t)x.v[2 * q + 1] << 16);
}
__device__ __forceinline__ void raw_from(Raw8<float>& f, const Frag<float>& x) {
#pragma unroll
    for (int q = 0; q < 8; ++q) f.w[q] = __float_as_uint(x.v[q]);
}

// Output element r (0..3) of lane l of a 16x16 accumulator sits at
// row 4*(l/16) + r, column l%16.
__device__ __forceinline__ int acc_row(int lane, int r) { return 4 * (lane >> 4) + r; }
__device__ __forceinline__ int acc_col(int lane) { return lane & 15; }

// ---------------------------------------------------------------------------
// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11)
struct u64x4 { uint64_t x[4]; };

__device__ __forceinline__ u64x4 philox4x64_10(u64x4 c, uint64_t k0, uint64_t k1) {
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        uint64_t lo0 = M0 * c.x[0], hi0 = __umul64hi(M0, c.x[0]);
        uint64_t lo1 = M1 * c.x[2], hi1 = __umul64hi(M1, c.x[2]);
        u64x4 n;
        n.x[0] = hi1 ^ c.x[1] ^ k0;
        n.x[1] = lo1;
        n.x[2] = hi0 ^ c.x[3] ^ k1;
        n.x[3] = lo0;
        c = n;
        k0 += W0;
        k1 += W1;
    }
    return c;
}

// ---------------------------------------------------------------------------
// Gate activations on the hardware exponential (v_exp_f32 via __expf) and
// reciprocal (v_rcp_f32).  sigmoid z = 1 / (1 + e^-z);  tanh z = 1 - 2 / (1 + e^{2z}),
// which saturates to +-1 without overflow (e^{2z} -> inf gives 1, -> 0 gives
// -1).  Absolute error a few 1e-7; the absolute error of tanh near 0 is that
// of 1 - (1 - 2z), i.e. about one float ulp of 1.
__device__ __forceinline__ float sigmoid_fast(float z) { return __builtin_amdgcn_rcpf(1.0f + __expf(-z)); }
__device__ __forceinline__ float tanh_fast(float z) { return 1.0f - 2.0f * __builtin_amdgcn_rcpf(1.0f + __expf(2.0f * z)); }

}  // namespace lsd
