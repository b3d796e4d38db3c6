// Internal interface between the C-ABI layer (pbb_api.cpp) and the HIP kernels
// (pbb_kernels.hip).  Not installed; not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pbb {

enum SupportMode : int32_t { kSupportPBB = 0, kSupportSWA = 1 };

// Largest number of (split, query head) states one unit of a split decode launch merges (the
// merge stages their maxima and sums in LDS).
constexpr int kMaxSplitStates = 2048;

constexpr int32_t kMaxGroup = 16;         // query heads per KV head held by one MFMA tile
constexpr int64_t kSplitMaxUnits = 64;    // bf16 decode launches with at most this many units split
constexpr int64_t kSplitMaxWays = 8;      // workgroups per unit of a split launch, at most
// bf16 decode launches with at most this many units over rings of at most this many slots
// prefetch the whole ring (one 32-slot chunk per wave of a 4-wave workgroup) at entry.
constexpr int32_t kWholeRingMaxUnits = 256;
constexpr int32_t kWholeRingMaxSlots = 128;
constexpr int kWholeRingWaves = 4;        // waves per workgroup of those launches

// Every decode workspace starts with a counter block of this size (one counter per unit of a
// split launch, at most kSplitMaxUnits), whatever the descriptor, so that one workspace,
// zero-filled once, serves split launches of every descriptor it is large enough for.
constexpr size_t kCounterBytes = 256;
static_assert(kCounterBytes >= (size_t)kSplitMaxUnits * 4, "counter block");

// Largest workspace a decode launch can need: the counter block, then the partial states of
// kSplitMaxUnits units (kSplitMaxWays splits x kMaxGroup heads x (head_dim 128 + maximum +
// sum) floats each) -- 4,260,096 bytes.  The allocation-free entry point keeps one buffer of
// this size per device.
constexpr size_t kNoAllocScratchBytes =
    kCounterBytes + (size_t)kSplitMaxUnits * kSplitMaxWays * kMaxGroup * (128 + 2) * 4;

// Everything a decode kernel needs, validated on the host before launch.
struct DecodeArgs {
  const int32_t* pos;
  int32_t* pos_next;   // optional: receives pos + 1 (pos itself for pos < 0); never aliases pos
  const void* q;
  const void* k_new;
  const void* v_new;
  void* k_ring;
  void* v_ring;
  void* out;
  int32_t batch;
  int32_t hq;
  int32_t hkv;
  int32_t group;       // query heads per KV head, 1..16
  int32_t slots;       // ring slots per (sequence, KV head)
  int32_t block;       // PBB block size B
  int32_t window;      // SWA window W
  int32_t mode;        // SupportMode
  float scale_log2;    // softmax scale times log2(e)
  int32_t rope;        // 1: rotate q and the new key by their position (rotary embedding)
  // Split of each unit's key steps over `splits` workgroups (1: none).  With splits > 1 the
  // workgroups of a unit leave partial states (unnormalised output, maximum and sum per head)
  // in ws_part and count in counters[unit]; the last to arrive merges them (Eq.(lse)) and
  // resets the counter to 0.
  int32_t splits;
  uint32_t* counters;  // [batch * hkv], zero between launches
  float* ws_part;      // [batch * hkv][splits][group][head_dim + 2]
  // Turns per position of rotary channel pair c (angle / 2 pi), c < head_dim / 2.
  double rope_turns[64];
};

// Prefill of prompts at positions 0..n-1, validated on the host before launch.
struct PrefillArgs {
  const void* q;       // [batch][n][hq][d]
  const void* k;       // [batch][n][hkv][d]
  const void* v;
  void* out;           // [batch][n][hq][d]
  float* lse;          // optional [batch][hq][n]
  void* k_ring;        // optional [batch][hkv][slots][d]
  void* v_ring;
  int32_t batch;
  int32_t n;
  int32_t hq;
  int32_t hkv;
  int32_t group;
  int32_t mode;        // SupportMode
  int32_t block;
  int32_t window;
  int32_t slots;
  float scale_log2;
};

// Backward of the prefill attention (gradients of q, k, v), validated on the host.
struct BackwardArgs {
  const void* q;       // [batch][n][hq][d]
  const void* k;       // [batch][n][hkv][d]
  const void* v;
  const void* out;     // forward output [batch][n][hq][d]
  const void* dout;    // upstream gradient [batch][n][hq][d]
  const float* lse;    // forward log-partitions (natural log) [batch][hq][n]
  void* dq;            // [batch][n][hq][d]
  void* dk;            // [batch][n][hkv][d]
  void* dv;
  float* ws;           // workspace [batch][hq][2][n]: lse * log2(e), then dout . out
  int32_t batch;
  int32_t n;
  int32_t hq;
  int32_t hkv;
  int32_t group;
  int32_t mode;        // SupportMode
  int32_t block;
  int32_t window;
  float scale;         // softmax scale
  float scale_log2;    // scale times log2(e)
};

hipError_t launch_ring_zero(void* k_ring, void* v_ring, size_t bytes_per_tensor,
                            hipStream_t stream);

hipError_t launch_ring_fill(const int32_t* pos, const void* k_src, const void* v_src,
                            void* k_ring, void* v_ring, int32_t batch, int32_t hkv,
                            int32_t src_len, int32_t slots, int32_t row_bytes,
                            hipStream_t stream);

// bf16 decode on matrix cores; head_dim 64 or 128.
hipError_t launch_decode_bf16(const DecodeArgs& a, int32_t head_dim, hipStream_t stream);

// bf16 prefill on matrix cores; head_dim 64 or 128; n >= 1.
hipError_t launch_prefill_bf16(const PrefillArgs& a, int32_t head_dim, hipStream_t stream);

// bf16 backward on matrix cores: delta, then dq, then dk/dv; head_dim 64 or 128; n >= 1.
hipError_t launch_backward_bf16(const BackwardArgs& a, int32_t head_dim, hipStream_t stream);

// fp32 decode on vector ALUs; head_dim 64 or 128.
hipError_t launch_decode_f32(const DecodeArgs& a, int32_t head_dim, hipStream_t stream);

// The library-held decode workspace of the current device (kNoAllocScratchBytes bytes): its
// device address, resolved once per device, whose first call also clears the counter block
// with a fill kernel on `stream`.  Allocates nothing.
hipError_t noalloc_scratch(void** ptr, hipStream_t stream);

}  // namespace pbb
