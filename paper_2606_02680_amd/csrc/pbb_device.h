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
// Largest sum of one lane's eight softmax weights of a column that a key step keeps without
// moving its reference: 2^8, so every weight stays <= 2^8, and a key whose score rises more
// than 8 log2 units above the reference (the usual dominant key of a peaked row) becomes the
// new reference and enters with weight exactly 1, unrounded.
constexpr float kWeightCap = 256.0f;

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

// First source a(t) of the support of target t: PBB (mode 0) max(0, h(floor(t/h) - 1)) with
// h = block/2 (Sec. 3 "Flash-PBB"), SWA max(0, t - window + 1) (Prop. 2).  Never decreases in t.
__device__ __forceinline__ int support_start(int mode, int block, int window, int t) {
  int lo;
  if (mode == 0) {
    const int h = block >> 1;
    lo = h * (t / h - 1);
  } else {
    lo = t - window + 1;
  }
  return lo > 0 ? lo : 0;
}

// Last target whose support contains source s (the largest t with support_start(t) <= s):
// PBB h(floor(s/h) + 2) - 1, SWA s + window - 1.
__device__ __forceinline__ int support_last_target(int mode, int block, int window, int s) {
  if (mode == 0) {
    const int h = block >> 1;
    return h * (s / h + 2) - 1;
  }
  return s + window - 1;
}

// Value of lane l ^ 16 and of lane l ^ 32 (gfx950 v_permlane16_swap / v_permlane32_swap with
// both operands x: one result is the lane's own value, the other its partner's), on the VALU
// instead of an LDS permute.
__device__ __forceinline__ float max_xor16_32(float x) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ float sum_xor16_32(float x) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// One 16-byte LDS DMA (global_load_lds) from a wave-uniform base plus a 32-bit lane offset, so
// that the address is formed by the instruction (scalar base + vector offset) rather than by
// 64-bit vector arithmetic.
__device__ __forceinline__ void dma16(const unsigned char* base, uint32_t off, unsigned char* lds) {
  __builtin_amdgcn_global_load_lds((const void*)(base + off),
                                   (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}

// Transposed LDS read (gfx950 ds_read_b64_tr_b16) at addr + OFF.  Issued as inline asm: the
// compiler cannot tell these reads apart from the LDS DMA still in flight and would otherwise
// wait for every outstanding load before each of them.  The caller waits with an s_waitcnt
// that takes the results as operands, so that nothing reads them earlier.
template <int OFF>
__device__ __forceinline__ u32x2 tr_read(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "LDS offset immediate");
  u32x2 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
  return r;
}

}  // namespace pbb
