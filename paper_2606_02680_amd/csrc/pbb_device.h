// Device-side helpers shared by the HIP kernels of libpbb (decode and prefill).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pbb {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;
typedef __attribute__((ext_vector_type(2))) unsigned int u32x2;

// Cache-policy operand of global_load_lds selecting the non-temporal ("nt") hint.
constexpr int kCachePolicyNT = 2;

constexpr float kNegInf = -__builtin_huge_valf();

// float -> bf16 with round-to-nearest-even (inputs are finite).
__device__ __forceinline__ uint16_t float_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Workgroup barrier that orders LDS reads and writes made by ordinary instructions, without
// waiting for LDS DMA still in flight (whose completion the caller tracks with vmcnt).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

}  // namespace pbb
