// The two 16-bit operand types of the matrix-core convolution kernels.
//
// Every kernel that multiplies 16-bit windows by the 16-bit packed filter is
// the same code for fp16 and bf16 operands: both are 2-byte elements that the
// transform, the filter pack and the LDS staging move as raw bits.  What
// differs is the 32x32x16 MFMA that consumes eight of them per lane and the
// rounding of the fp32 sums to the output type (nearest-even for both).
#pragma once

#include <stdint.h>

namespace im2win {

typedef float f32x16_acc __attribute__((ext_vector_type(16)));

// fp16 operands (IEEE binary16), v_mfma_f32_32x32x16_f16.
struct F16Op {
    typedef _Float16 v8 __attribute__((ext_vector_type(8)));
    typedef _Float16 elem;
    __device__ static inline f32x16_acc mfma(v8 a, v8 b, f32x16_acc c)
    {
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
    }
    // fp32 -> fp16 bits, round to nearest even
    __device__ static inline uint32_t bits(float x) { return __builtin_bit_cast(uint16_t, (_Float16)x); }
};

// bf16 operands (8-bit exponent, 8-bit significand), v_mfma_f32_32x32x16_bf16.
struct BF16Op {
    typedef __bf16 v8 __attribute__((ext_vector_type(8)));
    typedef __bf16 elem;
    __device__ static inline f32x16_acc mfma(v8 a, v8 b, f32x16_acc c)
    {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
    }
    // fp32 -> bf16 bits, round to nearest even (v_cvt_pk_bf16_f32)
    __device__ static inline uint32_t bits(float x) { return __builtin_bit_cast(uint16_t, (__bf16)x); }
};

}  // namespace im2win
