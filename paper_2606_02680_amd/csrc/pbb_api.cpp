// C ABI of libpbb (declared in include/pbb.h): argument validation, kernel selection and
// launch.  Every check runs on the host before anything is enqueued, so a failing call
// launches nothing and writes nothing.  No exception crosses the ABI.

#include "pbb.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "pbb_internal.h"

namespace {

static_assert(PBB_NOALLOC_SCRATCH_BYTES == pbb::kNoAllocScratchBytes,
              "the public scratch size must match the library's buffer");

using pbb::kMaxGroup;
using pbb::kSplitMaxUnits;
using pbb::kSplitMaxWays;
constexpr int32_t kMaxSlots = 65536;  // ring slots per (sequence, KV head)
constexpr int32_t kMaxPrefill = 1 << 30;  // prompt positions per call
constexpr int64_t kSplitUnits = 256;      // workgroups a split decode launch aims for (CUs)

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t elem_bytes(int32_t dtype) { return dtype == PBB_DTYPE_F32 ? 4 : 2; }

// Shape rules shared by every entry point; `swa` selects the sliding-window rules.
pbb_status_t check_desc(const pbb_desc_t* d, bool swa) {
  if (d == nullptr) return PBB_ERR_NULL;
  if (d->dtype != PBB_DTYPE_F32 && d->dtype != PBB_DTYPE_BF16) return PBB_ERR_DTYPE;
  if (d->batch < 1 || d->n_kv_heads < 1 || d->n_q_heads < 1) return PBB_ERR_SHAPE;
  if (d->n_q_heads % d->n_kv_heads != 0) return PBB_ERR_SHAPE;
  if (d->n_q_heads / d->n_kv_heads > kMaxGroup) return PBB_ERR_SHAPE;
  if (d->head_dim != 64 && d->head_dim != 128) return PBB_ERR_SHAPE;
  if (swa) {
    if (d->window < 1 || d->slots < d->window || d->slots > kMaxSlots) return PBB_ERR_SHAPE;
  } else {
    if (d->block < 2 || (d->block % 2) != 0 || d->block > kMaxSlots) return PBB_ERR_SHAPE;
    if (d->slots != d->block) return PBB_ERR_SHAPE;
  }
  if (!(d->rope_base == 0.0f || d->rope_base > 1.0f)) return PBB_ERR_SHAPE;  // NaN included
  // Ring element counts must fit comfortably in 64-bit offsets and the launch grid.
  const uint64_t rows = (uint64_t)d->batch * (uint64_t)d->n_kv_heads;
  if (rows > 0x7fffffffull) return PBB_ERR_SHAPE;
  return PBB_OK;
}

bool is_swa(const pbb_desc_t* d) { return d != nullptr && d->window > 0; }

size_t ring_tensor_bytes(const pbb_desc_t* d) {
  return (size_t)d->batch * (size_t)d->n_kv_heads * (size_t)d->slots * (size_t)d->head_dim *
         elem_bytes(d->dtype);
}

// Workgroups per (sequence, KV head) unit of a bf16 decode launch: launches with few units
// spread each unit's key steps over up to eight workgroups (at least eight 32-key steps each,
// two per wave of a 4-wave workgroup), so that more of the chip streams the rings.  The merge
// through the workspace costs a few serial device-coherent round trips (~2-3 us), which pays
// off for small batches with long supports.  The count is rounded down, so that a launch never
// exceeds one workgroup per CU (one more round of workgroups would double its time when the
// supports are equal, as in a full sliding window).
int32_t decode_splits(const pbb_desc_t* d, bool swa) {
  if (d->dtype != PBB_DTYPE_BF16) return 1;
  const int64_t units = (int64_t)d->batch * d->n_kv_heads;
  if (units > kSplitMaxUnits) return 1;
  const int64_t max_steps = ((int64_t)(swa ? d->window : d->block) + 31) / 32;
  int64_t s = std::min(kSplitUnits / units, (max_steps + 7) / 8);
  s = std::min<int64_t>(s, kSplitMaxWays);
  s = std::min<int64_t>(s, pbb::kMaxSplitStates / (d->n_q_heads / d->n_kv_heads));
  return (int32_t)std::max<int64_t>(1, s);
}

size_t decode_workspace(const pbb_desc_t* d, bool swa) {
  const int32_t s = decode_splits(d, swa);
  if (s <= 1) return 0;
  const size_t part = (size_t)d->batch * (size_t)d->n_kv_heads * (size_t)s *
                      (size_t)(d->n_q_heads / d->n_kv_heads) * (size_t)(d->head_dim + 2) * 4;
  return pbb::kCounterBytes + (part + 255) / 256 * 256;
}

// `use_scratch`: the workspace, when the launch needs one, is the library's per-device scratch
// buffer (the allocation-free entry point) instead of the caller's.
pbb_status_t decode_common(const pbb_desc_t* desc, bool swa, const int32_t* pos, int32_t* pos_next,
                           bool want_next, const void* q, const void* k_new, const void* v_new,
                           void* k_ring, void* v_ring, void* out, void* workspace,
                           size_t workspace_bytes, void* stream, bool use_scratch = false) {
  const pbb_status_t st = check_desc(desc, swa);
  if (st != PBB_OK) return st;
  if (!pos || !q || !k_new || !v_new || !k_ring || !v_ring || !out) return PBB_ERR_NULL;
  if (want_next && !pos_next) return PBB_ERR_NULL;
  if (want_next && !aligned(pos_next, 4)) return PBB_ERR_ALIGN;
  // pos_next must not overlap pos: other workgroups of the launch may still be reading pos.
  if (want_next && (const void*)pos_next < (const void*)(pos + desc->batch) &&
      (const void*)pos < (const void*)(pos_next + desc->batch))
    return PBB_ERR_SHAPE;
  if (!aligned(pos, 4) || !aligned(q, 16) || !aligned(k_new, 16) || !aligned(v_new, 16) ||
      !aligned(k_ring, 16) || !aligned(v_ring, 16) || !aligned(out, 16))
    return PBB_ERR_ALIGN;
  const size_t need = decode_workspace(desc, swa);
  if (use_scratch) {
    if (need > pbb::kNoAllocScratchBytes) return PBB_ERR_WORKSPACE;
    if (desc->rope_base > 0.0f && desc->dtype != PBB_DTYPE_BF16) return PBB_ERR_DTYPE;
    if (need > 0) {
      if (pbb::noalloc_scratch(&workspace, reinterpret_cast<hipStream_t>(stream)) != hipSuccess)
        return PBB_ERR_LAUNCH;
      workspace_bytes = pbb::kNoAllocScratchBytes;
    }
  }
  if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return PBB_ERR_WORKSPACE;
  if (need > 0 && !aligned(workspace, 16)) return PBB_ERR_ALIGN;

  pbb::DecodeArgs a;
  a.splits = need > 0 ? decode_splits(desc, swa) : 1;
  a.counters = need > 0 ? static_cast<uint32_t*>(workspace) : nullptr;
  a.ws_part = need > 0 ? reinterpret_cast<float*>(static_cast<unsigned char*>(workspace) +
                                                  pbb::kCounterBytes)
                       : nullptr;
  a.pos = pos;
  a.pos_next = want_next ? pos_next : nullptr;
  a.q = q;
  a.k_new = k_new;
  a.v_new = v_new;
  a.k_ring = k_ring;
  a.v_ring = v_ring;
  a.out = out;
  a.batch = desc->batch;
  a.hq = desc->n_q_heads;
  a.hkv = desc->n_kv_heads;
  a.group = desc->n_q_heads / desc->n_kv_heads;
  a.slots = desc->slots;
  a.block = desc->block;
  a.window = desc->window;
  a.mode = swa ? pbb::kSupportSWA : pbb::kSupportPBB;
  const float scale = desc->scale > 0.0f ? desc->scale
                                         : (float)(1.0 / std::sqrt((double)desc->head_dim));
  a.scale_log2 = (float)((double)scale * 1.4426950408889634);  // log2(e)
  a.rope = desc->rope_base > 0.0f ? 1 : 0;
  if (a.rope) {
    if (desc->dtype != PBB_DTYPE_BF16) return PBB_ERR_DTYPE;
    // Turns per position of channel pair c: base^(-2c/d) / (2 pi), in double.
    const double two_pi = 6.283185307179586476925286766559;
    for (int c = 0; c < desc->head_dim / 2; ++c)
      a.rope_turns[c] =
          std::pow((double)desc->rope_base, -2.0 * (double)c / (double)desc->head_dim) / two_pi;
    for (int c = desc->head_dim / 2; c < 64; ++c) a.rope_turns[c] = 0.0;
  } else {
    for (int c = 0; c < 64; ++c) a.rope_turns[c] = 0.0;
  }

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const hipError_t e = desc->dtype == PBB_DTYPE_BF16 ? pbb::launch_decode_bf16(a, desc->head_dim, s)
                                                     : pbb::launch_decode_f32(a, desc->head_dim, s);
  return e == hipSuccess ? PBB_OK : PBB_ERR_LAUNCH;
}

pbb_status_t prefill_common(const pbb_desc_t* desc, bool swa, int32_t n, const void* q,
                            const void* k, const void* v, void* out, float* lse, void* k_ring,
                            void* v_ring, void* stream) {
  const pbb_status_t st = check_desc(desc, swa);
  if (st != PBB_OK) return st;
  if (desc->dtype != PBB_DTYPE_BF16) return PBB_ERR_DTYPE;
  if (desc->rope_base != 0.0f) return PBB_ERR_SHAPE;  // prefill takes rotated inputs
  if (n < 0 || n > kMaxPrefill) return PBB_ERR_SHAPE;
  if (!q || !k || !v || !out) return PBB_ERR_NULL;
  if ((k_ring == nullptr) != (v_ring == nullptr)) return PBB_ERR_NULL;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
      !aligned(k_ring, 16) || !aligned(v_ring, 16) || !aligned(lse, 4))
    return PBB_ERR_ALIGN;
  // Workgroups: one per (sequence, KV head, tile of at least 8 positions).
  if ((uint64_t)desc->batch * (uint64_t)desc->n_kv_heads * ((uint64_t)n / 8 + 1) > 0x7fffffffull)
    return PBB_ERR_SHAPE;
  // 32 rows of one tensor lie within 32-bit byte offsets of the first
  if ((uint64_t)desc->n_q_heads * (uint64_t)desc->head_dim > (1u << 24)) return PBB_ERR_SHAPE;
  if (n == 0) return PBB_OK;

  pbb::PrefillArgs a;
  a.q = q;
  a.k = k;
  a.v = v;
  a.out = out;
  a.lse = lse;
  a.k_ring = k_ring;
  a.v_ring = v_ring;
  a.batch = desc->batch;
  a.n = n;
  a.hq = desc->n_q_heads;
  a.hkv = desc->n_kv_heads;
  a.group = desc->n_q_heads / desc->n_kv_heads;
  a.mode = swa ? pbb::kSupportSWA : pbb::kSupportPBB;
  a.block = desc->block;
  a.window = desc->window;
  a.slots = desc->slots;
  const float scale = desc->scale > 0.0f ? desc->scale
                                         : (float)(1.0 / std::sqrt((double)desc->head_dim));
  a.scale_log2 = (float)((double)scale * 1.4426950408889634);  // log2(e)
  const hipError_t e =
      pbb::launch_prefill_bf16(a, desc->head_dim, reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? PBB_OK : PBB_ERR_LAUNCH;
}

size_t backward_workspace(const pbb_desc_t* d, int32_t n) {
  const size_t f = (size_t)d->batch * (size_t)d->n_q_heads * (size_t)(n > 0 ? n : 0) * 8;
  return (f + 255) / 256 * 256;
}

pbb_status_t backward_common(const pbb_desc_t* desc, bool swa, int32_t n, const void* q,
                             const void* k, const void* v, const void* out, const void* dout,
                             const float* lse, void* dq, void* dk, void* dv, void* workspace,
                             size_t workspace_bytes, void* stream) {
  const pbb_status_t st = check_desc(desc, swa);
  if (st != PBB_OK) return st;
  if (desc->dtype != PBB_DTYPE_BF16) return PBB_ERR_DTYPE;
  if (desc->rope_base != 0.0f) return PBB_ERR_SHAPE;  // rotated inputs, as for prefill
  if (n < 0 || n > kMaxPrefill) return PBB_ERR_SHAPE;
  if (!q || !k || !v || !out || !dout || !lse || !dq || !dk || !dv) return PBB_ERR_NULL;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
      !aligned(dout, 16) || !aligned(dq, 16) || !aligned(dk, 16) || !aligned(dv, 16) ||
      !aligned(lse, 4))
    return PBB_ERR_ALIGN;
  if ((uint64_t)desc->batch * (uint64_t)desc->n_kv_heads * ((uint64_t)n / 4 + 1) > 0x7fffffffull)
    return PBB_ERR_SHAPE;
  // 32 rows of one tensor lie within 32-bit byte offsets of the first
  if ((uint64_t)desc->n_q_heads * (uint64_t)desc->head_dim > (1u << 24)) return PBB_ERR_SHAPE;
  // the delta launch covers 16 (d = 128) or 32 rows of batch x n x Hq per workgroup
  if ((uint64_t)desc->batch * (uint64_t)desc->n_q_heads * (uint64_t)n / 16 + 1 > 0x7fffffffull)
    return PBB_ERR_SHAPE;
  if (n == 0) return PBB_OK;
  if (workspace == nullptr || workspace_bytes < backward_workspace(desc, n))
    return PBB_ERR_WORKSPACE;
  if (!aligned(workspace, 16)) return PBB_ERR_ALIGN;

  pbb::BackwardArgs a;
  a.q = q;
  a.k = k;
  a.v = v;
  a.out = out;
  a.dout = dout;
  a.lse = lse;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  a.ws = static_cast<float*>(workspace);
  a.batch = desc->batch;
  a.n = n;
  a.hq = desc->n_q_heads;
  a.hkv = desc->n_kv_heads;
  a.group = desc->n_q_heads / desc->n_kv_heads;
  a.mode = swa ? pbb::kSupportSWA : pbb::kSupportPBB;
  a.block = desc->block;
  a.window = desc->window;
  a.scale = desc->scale > 0.0f ? desc->scale : (float)(1.0 / std::sqrt((double)desc->head_dim));
  a.scale_log2 = (float)((double)a.scale * 1.4426950408889634);
  const hipError_t e =
      pbb::launch_backward_bf16(a, desc->head_dim, reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? PBB_OK : PBB_ERR_LAUNCH;
}

}  // namespace

extern "C" {

const char* pbb_status_string(pbb_status_t status) {
  switch (status) {
    case PBB_OK: return "PBB_OK";
    case PBB_ERR_NULL: return "PBB_ERR_NULL: a required pointer is NULL";
    case PBB_ERR_SHAPE: return "PBB_ERR_SHAPE: inconsistent or unsupported sizes";
    case PBB_ERR_DTYPE: return "PBB_ERR_DTYPE: unsupported element type";
    case PBB_ERR_ALIGN: return "PBB_ERR_ALIGN: pointer not 16-byte aligned (pos: 4-byte)";
    case PBB_ERR_WORKSPACE: return "PBB_ERR_WORKSPACE: workspace too small";
    case PBB_ERR_LAUNCH: return "PBB_ERR_LAUNCH: the HIP runtime refused the launch";
  }
  return "PBB_ERR_UNKNOWN";
}

pbb_status_t pbb_ring_bytes(const pbb_desc_t* desc, size_t* bytes_per_tensor) {
  if (desc == nullptr || bytes_per_tensor == nullptr) return PBB_ERR_NULL;
  const pbb_status_t st = check_desc(desc, is_swa(desc));
  if (st != PBB_OK) return st;
  *bytes_per_tensor = ring_tensor_bytes(desc);
  return PBB_OK;
}

pbb_status_t pbb_ring_init(const pbb_desc_t* desc, void* k_ring, void* v_ring, void* stream) {
  const pbb_status_t st = check_desc(desc, is_swa(desc));
  if (st != PBB_OK) return st;
  if (!k_ring || !v_ring) return PBB_ERR_NULL;
  if (!aligned(k_ring, 16) || !aligned(v_ring, 16)) return PBB_ERR_ALIGN;
  const hipError_t e = pbb::launch_ring_zero(k_ring, v_ring, ring_tensor_bytes(desc),
                                             reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? PBB_OK : PBB_ERR_LAUNCH;
}

pbb_status_t pbb_ring_fill(const pbb_desc_t* desc, const int32_t* pos, const void* k_src,
                           const void* v_src, int32_t src_len, void* k_ring, void* v_ring,
                           void* stream) {
  const pbb_status_t st = check_desc(desc, is_swa(desc));
  if (st != PBB_OK) return st;
  if (src_len < 0 || src_len > desc->slots) return PBB_ERR_SHAPE;
  if (!pos || !k_ring || !v_ring) return PBB_ERR_NULL;
  if (src_len > 0 && (!k_src || !v_src)) return PBB_ERR_NULL;
  if (!aligned(pos, 4) || !aligned(k_ring, 16) || !aligned(v_ring, 16) ||
      (src_len > 0 && (!aligned(k_src, 16) || !aligned(v_src, 16))))
    return PBB_ERR_ALIGN;
  const int32_t row_bytes = desc->head_dim * (int32_t)elem_bytes(desc->dtype);
  const hipError_t e = pbb::launch_ring_fill(pos, k_src, v_src, k_ring, v_ring, desc->batch,
                                             desc->n_kv_heads, src_len, desc->slots, row_bytes,
                                             reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? PBB_OK : PBB_ERR_LAUNCH;
}

pbb_status_t pbb_workspace_bytes(const pbb_desc_t* desc, size_t* bytes) {
  if (desc == nullptr || bytes == nullptr) return PBB_ERR_NULL;
  const pbb_status_t st = check_desc(desc, false);
  if (st != PBB_OK) return st;
  *bytes = decode_workspace(desc, false);
  return PBB_OK;
}

pbb_status_t swa_workspace_bytes(const pbb_desc_t* desc, size_t* bytes) {
  if (desc == nullptr || bytes == nullptr) return PBB_ERR_NULL;
  const pbb_status_t st = check_desc(desc, true);
  if (st != PBB_OK) return st;
  *bytes = decode_workspace(desc, true);
  return PBB_OK;
}

pbb_status_t pbb_decode_step(const pbb_desc_t* desc, const int32_t* pos, const void* q,
                             const void* k_new, const void* v_new, void* k_ring, void* v_ring,
                             void* out, void* workspace, size_t workspace_bytes, void* stream) {
  return decode_common(desc, false, pos, nullptr, false, q, k_new, v_new, k_ring, v_ring, out,
                       workspace, workspace_bytes, stream);
}

pbb_status_t swa_decode_step(const pbb_desc_t* desc, const int32_t* pos, const void* q,
                             const void* k_new, const void* v_new, void* k_ring, void* v_ring,
                             void* out, void* workspace, size_t workspace_bytes, void* stream) {
  return decode_common(desc, true, pos, nullptr, false, q, k_new, v_new, k_ring, v_ring, out,
                       workspace, workspace_bytes, stream);
}

pbb_status_t pbb_decode_step_noalloc(const pbb_desc_t* desc, const int32_t* pos, const void* q,
                                     const void* k_new, const void* v_new, void* k_ring,
                                     void* v_ring, void* out, void* stream) {
  return decode_common(desc, false, pos, nullptr, false, q, k_new, v_new, k_ring, v_ring, out,
                       nullptr, 0, stream, true);
}

pbb_status_t pbb_decode_step_advance(const pbb_desc_t* desc, const int32_t* pos, int32_t* pos_next,
                                     const void* q, const void* k_new, const void* v_new,
                                     void* k_ring, void* v_ring, void* out, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  return decode_common(desc, false, pos, pos_next, true, q, k_new, v_new, k_ring, v_ring, out,
                       workspace, workspace_bytes, stream);
}

pbb_status_t swa_decode_step_advance(const pbb_desc_t* desc, const int32_t* pos, int32_t* pos_next,
                                     const void* q, const void* k_new, const void* v_new,
                                     void* k_ring, void* v_ring, void* out, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  return decode_common(desc, true, pos, pos_next, true, q, k_new, v_new, k_ring, v_ring, out,
                       workspace, workspace_bytes, stream);
}

pbb_status_t pbb_prefill(const pbb_desc_t* desc, int32_t n, const void* q, const void* k,
                         const void* v, void* out, float* lse, void* k_ring, void* v_ring,
                         void* stream) {
  return prefill_common(desc, false, n, q, k, v, out, lse, k_ring, v_ring, stream);
}

pbb_status_t swa_prefill(const pbb_desc_t* desc, int32_t n, const void* q, const void* k,
                         const void* v, void* out, float* lse, void* k_ring, void* v_ring,
                         void* stream) {
  return prefill_common(desc, true, n, q, k, v, out, lse, k_ring, v_ring, stream);
}

pbb_status_t pbb_backward_workspace_bytes(const pbb_desc_t* desc, int32_t n, size_t* bytes) {
  if (desc == nullptr || bytes == nullptr) return PBB_ERR_NULL;
  const pbb_status_t st = check_desc(desc, is_swa(desc));
  if (st != PBB_OK) return st;
  if (n < 0 || n > kMaxPrefill) return PBB_ERR_SHAPE;
  *bytes = backward_workspace(desc, n);
  return PBB_OK;
}

pbb_status_t pbb_backward(const pbb_desc_t* desc, int32_t n, const void* q, const void* k,
                          const void* v, const void* out, const void* dout, const float* lse,
                          void* dq, void* dk, void* dv, void* workspace, size_t workspace_bytes,
                          void* stream) {
  return backward_common(desc, false, n, q, k, v, out, dout, lse, dq, dk, dv, workspace,
                         workspace_bytes, stream);
}

pbb_status_t swa_backward(const pbb_desc_t* desc, int32_t n, const void* q, const void* k,
                          const void* v, const void* out, const void* dout, const float* lse,
                          void* dq, void* dk, void* dv, void* workspace, size_t workspace_bytes,
                          void* stream) {
  return backward_common(desc, true, n, q, k, v, out, dout, lse, dq, dk, dv, workspace,
                         workspace_bytes, stream);
}

}  // extern "C"
