// device_math.hpp -- element formats and fp32 math shared by the gfx950 scan kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mbs {

// Native vector types (clang ext vectors: usable with the nontemporal builtins).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;  // log2(e)
constexpr float kLn2 = 0.6931471805599453f;    // ln(2)

// bfloat16 is the upper half of an IEEE float: widening is a shift.
__device__ __forceinline__ float bf16_lo(uint32_t pair) { return __uint_as_float(pair << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t pair) { return __uint_as_float(pair & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Round to nearest even.  A NaN stays a NaN (quiet, sign kept): adding the
// rounding bias to a NaN with its high mantissa bits set would carry into the
// exponent and sign and turn it into a zero.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t x = __float_as_uint(f);
    if ((x & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((x >> 16) | 0x40u);
    x += 0x7fffu + ((x >> 16) & 1u);
    return (uint16_t)(x >> 16);
}

// Two floats rounded to bfloat16 and packed, a in the low half: one
// v_cvt_pk_bf16_f32 on gfx950.  It rounds to nearest even and keeps a NaN a quiet
// NaN with its sign, so it gives f32_to_bf16's bits for every fp32 pattern
// (bf16_pack_check.hip compares the two over all 2^32 of them on the GPU).
__device__ __forceinline__ uint32_t bf16x2_pack(float a, float b) {
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
}

// Hardware transcendentals: v_exp_f32 = 2^x, v_log_f32 = log2 x, v_rcp_f32 = 1/x.
__device__ __forceinline__ float hw_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float hw_log2(float x) { return __builtin_amdgcn_logf(x); }
__device__ __forceinline__ float hw_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

// softplus(v) = log(1 + e^v), the positivity map of the timestep (eq. (3)),
// as max(v, 0) + log1p(e) with e = e^-|v| in (0, 1].  log1p(e) is taken as
// log(w) with w = fl(1 + e) in [1, 2], plus the rounding error c = e - (w - 1)
// (exact in fp32 by Sterbenz) divided by w; using c for c / w leaves an error
// of at most c * e <= 2^-24 * e, i.e. relative 2^-24, so the result is
// accurate to a few ulp for every v, including large negative v where the
// naive log(1 + e^v) loses all digits.
__device__ __forceinline__ float softplus_f32(float v) {
    const float e = hw_exp2(-__builtin_fabsf(v) * kLog2e);
    const float w = 1.0f + e;
    const float c = e - (w - 1.0f);
    return __builtin_fmaxf(v, 0.0f) + __builtin_fmaf(hw_log2(w), kLn2, c);
}

// silu(z) = z * sigmoid(z), the Swish gate (Table 8, Fig. 5).
__device__ __forceinline__ float silu_f32(float z) {
    return z * hw_rcp(1.0f + hw_exp2(-z * kLog2e));
}

template <int DT> struct Act;  // element access by mb_dtype

template <> struct Act<0> {    // MB_F32
    using T = float;
    static __device__ __forceinline__ float ld(const void *p, int64_t i) {
        return static_cast<const float *>(p)[i];
    }
};
template <> struct Act<1> {    // MB_BF16
    using T = uint16_t;
    static __device__ __forceinline__ float ld(const void *p, int64_t i) {
        return bf16_to_f32(static_cast<const uint16_t *>(p)[i]);
    }
};

template <int DT> __device__ __forceinline__ void st_out(void *p, int64_t i, float v);
template <> __device__ __forceinline__ void st_out<0>(void *p, int64_t i, float v) {
    static_cast<float *>(p)[i] = v;
}
template <> __device__ __forceinline__ void st_out<1>(void *p, int64_t i, float v) {
    static_cast<uint16_t *>(p)[i] = f32_to_bf16(v);
}

}  // namespace mbs
