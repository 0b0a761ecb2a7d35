// zq_device.h -- device helpers shared by the codec kernels and the
// dequantising GEMM: vector types, bit casts and the binary32 -> bf16 / fp16
// narrowings (nearest even) used wherever a dequantised value is stored.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace zq {

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t f2u(float f) { return __builtin_bit_cast(uint32_t, f); }
__device__ __forceinline__ float u2f(uint32_t u) { return __builtin_bit_cast(float, u); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// two binary32 -> two bfloat16 (v_cvt_pk_bf16_f32, nearest even)
__device__ __forceinline__ uint32_t bf16x2_bits(float a, float b) {
  f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

__device__ __forceinline__ float h2f(uint32_t bits16) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}
// binary32 -> binary16, nearest even (v_cvt_f16_f32).  The empty asm pins v
// as a materialised binary32 value: without it the compiler folds a preceding
// fp32 multiply and this narrowing into one v_fma_mixlo_f16, which rounds the
// exact product once instead of rounding it to binary32 first.
__device__ __forceinline__ uint32_t f2h(float v) {
  asm("" : "+v"(v));
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)v);
}

}  // namespace zq
