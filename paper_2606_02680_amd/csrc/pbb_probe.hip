// Streaming-read probe (libpbbprobe): the LDS-DMA streaming skeleton of the bf16 decode kernel
// without its arithmetic, used to measure the practical HBM read rate of the decode's access
// pattern.  See include/pbb_probe.h.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pbb_device.h"
#include "pbb_probe.h"

namespace {

constexpr int kRowBytes = 256;            // one bf16 row of head_dim 128
constexpr int kStepRows = 32;             // rows of K (and of V) per wave step
constexpr int kTile = kStepRows * kRowBytes;   // 8 KiB
constexpr int kOps = 2 * kTile / 1024;    // 16 DMA instructions (1 KiB each) per step

template <int NW, bool NT>
__global__ __launch_bounds__(NW * 64) void stream_probe_kernel(const unsigned char* __restrict__ k,
                                                               const unsigned char* __restrict__ v,
                                                               size_t unit_stride,
                                                               const int32_t* __restrict__ rows,
                                                               int max_rows, float* sink) {
  __shared__ __align__(16) unsigned char lds[NW][2][2 * kTile];
  const int u = blockIdx.x;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n = min(max(rows[u], 0), max_rows);
  const int nsteps = (n + kStepRows - 1) / kStepRows;
  const unsigned char* kb = k + (size_t)u * unit_stride;
  const unsigned char* vb = v + (size_t)u * unit_stride;
  // Lane l moves 16-byte piece l % 16 of row 4x + l / 16 of the step (x < 8) for each tensor.
  auto issue = [&](int buf, int step) {
    unsigned char* t = &lds[wave][buf][0];
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      const int row = step * kStepRows + 4 * x + lane / 16;
      const int r = row < n ? row : 0;          // past the end: row 0 (in bounds, unused)
      const size_t off = (size_t)r * kRowBytes + (lane % 16) * 16;
      __builtin_amdgcn_global_load_lds((const void*)(kb + off),
                                       (__attribute__((address_space(3))) void*)(t + x * 1024),
                                       16, 0, NT ? pbb::kCachePolicyNT : 0);
      __builtin_amdgcn_global_load_lds((const void*)(vb + off),
                                       (__attribute__((address_space(3))) void*)(t + kTile + x * 1024),
                                       16, 0, NT ? pbb::kCachePolicyNT : 0);
    }
  };
  float acc = 0.0f;
  int step = wave;
  issue(0, step);
  issue(1, step + NW);
  int buf = 0;
  for (; step < nsteps; step += NW) {
    // this step's tiles have landed once at most the next step's kOps loads are outstanding
    __builtin_amdgcn_s_waitcnt(0x0F70 | (kOps & 15) | ((kOps >> 4) << 14));
    __builtin_amdgcn_sched_barrier(0);
    acc += *(const float*)&lds[wave][buf][lane * 16];
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    issue(buf, step + 2 * NW);
    buf ^= 1;
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);   // drain the trailing prefetches
  if (acc == 1.2345678f) sink[0] = acc;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

extern "C" int pbb_probe_stream(const void* k, const void* v, size_t unit_stride,
                                const int32_t* rows, int32_t units, int32_t max_rows,
                                int32_t waves, int32_t nontemporal, float* sink, void* stream) {
  if (!k || !v || !rows || !sink || units < 1 || max_rows < 1 || (waves != 2 && waves != 4))
    return 1;
  if ((size_t)max_rows * kRowBytes > unit_stride || !aligned16(k) || !aligned16(v) ||
      (unit_stride & 15u) != 0)
    return 1;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const dim3 grid((unsigned)units);
  const auto* kk = static_cast<const unsigned char*>(k);
  const auto* vv = static_cast<const unsigned char*>(v);
  if (waves == 4) {
    if (nontemporal) hipLaunchKernelGGL((stream_probe_kernel<4, true>), grid, dim3(256), 0, s, kk, vv, unit_stride, rows, max_rows, sink);
    else hipLaunchKernelGGL((stream_probe_kernel<4, false>), grid, dim3(256), 0, s, kk, vv, unit_stride, rows, max_rows, sink);
  } else {
    if (nontemporal) hipLaunchKernelGGL((stream_probe_kernel<2, true>), grid, dim3(128), 0, s, kk, vv, unit_stride, rows, max_rows, sink);
    else hipLaunchKernelGGL((stream_probe_kernel<2, false>), grid, dim3(128), 0, s, kk, vv, unit_stride, rows, max_rows, sink);
  }
  return (int)hipGetLastError();
}
