// Shared device-side types and helpers of the PCPP HIP library (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pcpp {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// One 32x32x16 bf16 MFMA: acc (32x32 fp32) += A (32x16) * B (16x32).
// Operand lane layout: lane l holds row/column (l % 32) and one half
// (l / 32) of the 16-long contraction; the output holds column (l % 32) and
// rows 8*(r/4) + 4*(l/32) + (r%4) in register r.
__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 acc) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
}

__device__ __forceinline__ float bf16_to_f32(bf16 x) { return (float)x; }
__device__ __forceinline__ bf16 f32_to_bf16(float x) { return (bf16)x; }  // RNE

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

}  // namespace pcpp
