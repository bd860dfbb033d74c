// fa_common.h -- device-side helpers shared by the gfx950 attention kernels.
//
// Lane layouts of the matrix instructions used here (checked on gfx950):
//   v_mfma_f32_32x32x16_{f16,bf16}: A lane l holds A[l%32][8*(l/32)+e],
//     B lane l holds B[8*(l/32)+e][l%32] (e = 0..7), C lane l register r holds
//     C[8*(r/4) + 4*(l/32) + r%4][l%32] (r = 0..15).
//   v_mfma_f32_16x16x32_{f16,bf16}: A lane l holds A[l%16][8*(l/16)+e],
//     B lane l holds B[8*(l/16)+e][l%16], C lane l register r holds
//     C[4*(l/16)+r][l%16] (r = 0..3).
//   ds_read_b64_tr_b16: within each group of 16 lanes, result element e of
//     lane j is element j%4 of the 8 bytes addressed by lane 4*e + j/4.  So if
//     lane i of the group addresses row (r0 + i/4), columns c0 + 4*(i%4)..+3 of
//     a row-major 16-bit matrix, lane j receives column c0 + j of rows r0..r0+3.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fa {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short short4_t __attribute__((ext_vector_type(4)));
typedef float float16_t __attribute__((ext_vector_type(16)));
typedef float float4_t __attribute__((ext_vector_type(4)));
typedef unsigned int uint4_t __attribute__((ext_vector_type(4)));

// Storage types as seen by the kernels.
struct f16_t {
    typedef _Float16 scalar;
    typedef half8_t vec8;
};
struct bf16_t {
    typedef __bf16 scalar;
    typedef bf16x8_t vec8;
};

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// 16-bit storage word -> fp32 (exact for both formats).
__device__ __forceinline__ float to_f32(_Float16 x) { return (float)x; }
__device__ __forceinline__ float to_f32(__bf16 x) { return (float)x; }
__device__ __forceinline__ float to_f32(float x) { return x; }

// fp32 -> output element, round to nearest even.
template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ _Float16 from_f32<_Float16>(float x) { return (_Float16)x; }
template <> __device__ __forceinline__ __bf16 from_f32<__bf16>(float x) { return (__bf16)x; }

// Matrix instruction wrappers, one per input element type.
__device__ __forceinline__ float16_t mfma32(half8_t a, half8_t b, float16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ float16_t mfma32(bf16x8_t a, bf16x8_t b, float16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ float4_t mfma16(half8_t a, half8_t b, float4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ float4_t mfma16(bf16x8_t a, bf16x8_t b, float4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Eight 16-bit values loaded / stored as one 16-byte word.
template <typename V> __device__ __forceinline__ V as_vec8(uint4_t u) {
    return __builtin_bit_cast(V, u);
}
template <typename V> __device__ __forceinline__ uint4_t as_u4(V v) {
    return __builtin_bit_cast(uint4_t, v);
}

// bf16 x8 (as raw 16-byte word) -> f16 x8 (raw), round to nearest even.
__device__ __forceinline__ uint4_t bf16x8_to_f16x8(uint4_t u) {
    half8_t h;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        h[2 * i] = (_Float16)__uint_as_float(u[i] << 16);
        h[2 * i + 1] = (_Float16)__uint_as_float(u[i] & 0xffff0000u);
    }
    return __builtin_bit_cast(uint4_t, h);
}

// Two fp32 values -> packed f16 pair (first in the low half), round to nearest even.
__device__ __forceinline__ unsigned pack_f16x2(float lo, float hi) {
    half2_t h;
    h[0] = (_Float16)lo;
    h[1] = (_Float16)hi;
    return __builtin_bit_cast(unsigned, h);
}

// Pack 8 fp32 values to f16 x8, round to nearest even.
__device__ __forceinline__ half8_t pack_f16x8(float a0, float a1, float a2, float a3, float a4,
                                              float a5, float a6, float a7) {
    half8_t h;
    h[0] = (_Float16)a0; h[1] = (_Float16)a1; h[2] = (_Float16)a2; h[3] = (_Float16)a3;
    h[4] = (_Float16)a4; h[5] = (_Float16)a5; h[6] = (_Float16)a6; h[7] = (_Float16)a7;
    return h;
}

// Sum of 16 f16 values (two f16 x8 words) accumulated in fp32 (dot products
// with (1, 1), two independent chains).
__device__ __forceinline__ float sum_f16x16(half8_t a, half8_t b) {
    const half2_t one = {(_Float16)1.0f, (_Float16)1.0f};
    float s0 = 0.f, s1 = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        s0 = __builtin_amdgcn_fdot2(half2_t{a[2 * i], a[2 * i + 1]}, one, s0, false);
        s1 = __builtin_amdgcn_fdot2(half2_t{b[2 * i], b[2 * i + 1]}, one, s1, false);
    }
    return s0 + s1;
}

// Reductions over the lane pair (l, l^32).  v_permlane32_swap exchanges the
// upper half of its first operand with the lower half of its second; with the
// same value in both, the two results of every lane are the pair's two values
// (one from each half), whichever result holds which.
__device__ __forceinline__ float pair_max(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                              false);
    return __builtin_fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                              false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float max3(float a, float b, float c) {
    return __builtin_fmaxf(a, __builtin_fmaxf(b, c));
}

// LDS transpose read (see the layout note at the top of this file).
__device__ __forceinline__ short4_t lds_read_tr16(const _Float16 *p) {
    typedef __attribute__((address_space(3))) short4_t lds_s4;
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4 *)(p));
}

__device__ __forceinline__ half8_t cat_half8(short4_t lo, short4_t hi) {
    typedef short short8_t __attribute__((ext_vector_type(8)));
    short8_t s = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(half8_t, s);
}

// Global 16-byte load / store helpers.
__device__ __forceinline__ uint4_t ld16(const void *p) {
    return *reinterpret_cast<const uint4_t *>(p);
}
__device__ __forceinline__ void st16(void *p, uint4_t v) { *reinterpret_cast<uint4_t *>(p) = v; }
// Streaming 16-byte load for data read exactly once (non-temporal hint).
__device__ __forceinline__ uint4_t ld16_stream(const void *p) {
    return __builtin_nontemporal_load(reinterpret_cast<const uint4_t *>(p));
}

}  // namespace fa
