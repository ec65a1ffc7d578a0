// Device-side helpers shared by the gfx950 kernels: vector types, bf16
// conversion, buffer-resource loads and the MFMA operand conventions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace isam {

// Compile-time loop: f(std::integral_constant<int, I>{}) for I = 0 .. N-1, so
// register-array indices stay constants (no dynamic indexing into scratch).
template <int I, int N>
struct StaticFor {
    template <typename F>
    __device__ __forceinline__ static void run(F&& f) {
        f(std::integral_constant<int, I>{});
        StaticFor<I + 1, N>::run(f);
    }
};
template <int N>
struct StaticFor<N, N> {
    template <typename F>
    __device__ __forceinline__ static void run(F&&) {}
};
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    StaticFor<0, N>::run(f);
}

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(4))) int i32x4_t;

typedef uint16_t bf16_t;  // bf16 stored as its 16-bit pattern

// ---------------------------------------------------------------------------
// bf16 <-> fp32
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}
__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Round to nearest, ties to even (inputs here are finite).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return f32_to_bf16(lo) | (f32_to_bf16(hi) << 16);
}

// fp32 as the sum of three bf16 terms: h = bf16(x), m = bf16(x - h),
// l = bf16(x - h - m) (each difference is exact in fp32; |x - h - m - l| is
// at most 2^-24 |x|).  A product a.b to fp32 accuracy is then the six bf16
// products hh + hm + mh + hl + lh + mm, every one exact in fp32 (the dropped
// ml, lm, ll are below 2^-23 |a.b|).
typedef __bf16 f32s_bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32s_f32x2_t __attribute__((ext_vector_type(2)));
// Two fp32 values to a bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16_rne(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32s_f32x2_t){lo, hi}, f32s_bf16x2_t));
}
// The three bf16 terms of two fp32 values, as packed pairs t[0] (h), t[1] (m), t[2] (l).
__device__ __forceinline__ void split3_pair(float x0, float x1, uint32_t t[3]) {
    t[0] = pack_bf16_rne(x0, x1);
    const float r0 = x0 - __uint_as_float(t[0] << 16), r1 = x1 - __uint_as_float(t[0] & 0xffff0000u);
    t[1] = pack_bf16_rne(r0, r1);
    const float q0 = r0 - __uint_as_float(t[1] << 16), q1 = r1 - __uint_as_float(t[1] & 0xffff0000u);
    t[2] = pack_bf16_rne(q0, q1);
}

// ---------------------------------------------------------------------------
// Buffer resources: a raw (stride 0) buffer whose loads past num_records
// bytes return zero.  Used for ragged tile edges: an out-of-range element is
// addressed at an offset beyond the record count instead of being branched
// around.
// ---------------------------------------------------------------------------
constexpr int kBufferFlags = 0x00020000;  // gfx9 data format word
constexpr uint32_t kOob = 0x80000000u;    // offset guaranteed beyond num_records

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                             kBufferFlags);
}
__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    i32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
    return __builtin_bit_cast(uint4, v);
}
__device__ __forceinline__ uint32_t buf_load4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0);
}
__device__ __forceinline__ uint32_t buf_load2(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, 0);
}

// ---------------------------------------------------------------------------
// MFMA wrappers.  Operand convention used by every kernel in this library:
//   32x32 tiles: lane l supplies row (l % 32) of A and column (l % 32) of B;
//   the lane half g = l / 32 selects which K sub-range the lane carries.
//   Each lane carries 16 contiguous bytes of K per operand: 8 bf16 (one
//   32x32x16 instruction) or 4 fp32 (four 32x32x2 instructions, element e
//   of the chunk going to instruction e).  A and B use the same K assignment,
//   so the contraction is exact in any K order.
//   Accumulator element v of lane l is C[8*(v/4) + 4*(l/32) + (v%4)][l % 32].
// ---------------------------------------------------------------------------
__device__ __forceinline__ void mfma32_bf16(f32x16_t& acc, uint4 a, uint4 b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                  __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
}
__device__ __forceinline__ void mfma32_f32x4(f32x16_t& acc, uint4 a, uint4 b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
}
// 16x16 tiles: lane l supplies row (l % 16) of A / column (l % 16) of B, the
// lane quarter l / 16 selects the K sub-range; accumulator element v of lane l
// is C[4*(l/16) + v][l % 16].
__device__ __forceinline__ void mfma16_bf16(f32x4_t& acc, uint4 a, uint4 b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                  __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
}
__device__ __forceinline__ void mfma16_f32x4(f32x4_t& acc, uint4 a, uint4 b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// In-register transposes used when an operand is stored with M (or N)
// contiguous: a thread loads E rows of K (16 bytes each, E elements along M/N)
// and turns them into E chunks of E consecutive K values, one per M/N index.
// ---------------------------------------------------------------------------
// 8x8 of 16-bit elements: in[r] holds row r (elements 2p, 2p+1 in word p);
// out[c] word p = (in[2p][c] in the low half, in[2p+1][c] in the high half).
__device__ __forceinline__ void transpose8x8_b16(const uint4 in[8], uint4 out[8]) {
    uint32_t w[8][4];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
        w[r][0] = in[r].x; w[r][1] = in[r].y; w[r][2] = in[r].z; w[r][3] = in[r].w;
    }
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        uint32_t o[4];
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            uint32_t lo = w[2 * p][c >> 1], hi = w[2 * p + 1][c >> 1];
            o[p] = (c & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
        }
        out[c] = make_uint4(o[0], o[1], o[2], o[3]);
    }
}
// 4x4 of 32-bit elements.
__device__ __forceinline__ void transpose4x4_b32(const uint4 in[4], uint4 out[4]) {
    out[0] = make_uint4(in[0].x, in[1].x, in[2].x, in[3].x);
    out[1] = make_uint4(in[0].y, in[1].y, in[2].y, in[3].y);
    out[2] = make_uint4(in[0].z, in[1].z, in[2].z, in[3].z);
    out[3] = make_uint4(in[0].w, in[1].w, in[2].w, in[3].w);
}

}  // namespace isam
