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

// Rotary embedding of one channel pair at absolute position t: the angle in turns,
// t * turns_per_pos, is reduced to [0, 1) in fp64 (exact enough for any t < 2^31) and the
// hardware sine and cosine (which take turns) give cos and sin.
__device__ __forceinline__ void rope_cos_sin(int t, double turns_per_pos, float& cs, float& sn) {
  const double r = (double)t * turns_per_pos;
  const float f = (float)(r - __builtin_floor(r));
  cs = __builtin_amdgcn_cosf(f);
  sn = __builtin_amdgcn_sinf(f);
}

// (x, y) = channels (c, c + d/2) turned by the angle: (x cos - y sin, y cos + x sin), with the
// same fused operations wherever it is evaluated.
__device__ __forceinline__ void rope_turn(float x, float y, float cs, float sn, float& ox,
                                          float& oy) {
  ox = __builtin_fmaf(x, cs, -(y * sn));
  oy = __builtin_fmaf(y, cs, x * sn);
}

// Workgroup barrier that orders LDS reads and writes made by ordinary instructions, without
// waiting for LDS DMA still in flight (whose completion the caller tracks with vmcnt).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

}  // namespace pbb
