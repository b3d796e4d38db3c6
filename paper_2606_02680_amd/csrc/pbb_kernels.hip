// HIP kernels for Post-Boundary Bridge (PBB) decode on gfx950 (MI355X, CDNA4).
//
// One decode step for a (sequence, KV head) pair reads the support of t = pos[b] straight
// from the ring, in slot space.  With h = B/2 the PBB support is the interval
// [a(t), t], a(t) = max(0, h*(floor(t/h) - 1)) (Sec. 3 "Flash-PBB"; Appendix A.3,
// Eq.(pbb_relay)); since position s lives at slot s mod B, the sources other than t occupy
//   slots [h, B)  (positions p-h .. p-1)   when p > 0 and r < h   (the bridge), then
//   slots [0, r)  (positions p .. t-1)                           (the block prefix)
// (Appendix F.1, the paragraph after the ring proposition).  The sliding-window baseline
// reads positions max(0, t-W+1) .. t-1, i.e. one slot range modulo S that may wrap once.
// Both are described below as "ring key i of n_ring": slot = base0 + i for i < len0, else
// i - len0.  The current token t is one extra key taken from k_new/v_new, never from the
// ring, and the same launch writes it into slot t mod slots, which holds t - slots: a
// position outside the support (Appendix F.1, proof of the proposition), so no read in the
// launch can observe the write.
//
// Softmax: scores are q.k * scale; exponentials are taken base 2 on scores pre-multiplied by
// log2(e), with a running maximum (online softmax) and fp32 accumulation (Eq.(attention)).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pbb_device.h"
#include "pbb_internal.h"

namespace pbb {
namespace {

// Ring-key ranges of one (sequence, KV head) at position t.
struct Ranges {
  int n_ring;       // sources read from the ring (the support minus t itself)
  int len0;         // length of the first slot range
  int base0;        // first slot of the first range; the second range starts at slot 0
  int append_slot;  // slot that receives position t
};

__device__ __forceinline__ Ranges pbb_ranges(int t, int block) {
  const int h = block >> 1;
  const int r = t % block;
  const int p = t - r;
  const bool bridge = (p > 0) && (r < h);  // Eq.(pbb): bridge only after block 0, r < h
  Ranges R;
  R.len0 = bridge ? h : 0;
  R.base0 = h;
  R.n_ring = R.len0 + r;
  R.append_slot = r;
  return R;
}

__device__ __forceinline__ Ranges swa_ranges(int t, int window, int slots) {
  const int s0 = max(0, t - window + 1);  // Prop. 2: the window includes t
  Ranges R;
  R.n_ring = t - s0;
  R.base0 = s0 % slots;
  R.len0 = min(R.n_ring, slots - R.base0);
  R.append_slot = t % slots;
  return R;
}

__device__ __forceinline__ Ranges ranges_for(const DecodeArgs& a, int t) {
  return a.mode == kSupportPBB ? pbb_ranges(t, a.block) : swa_ranges(t, a.window, a.slots);
}

__device__ __forceinline__ int ring_slot(const Ranges& R, int i) {
  return i < R.len0 ? R.base0 + i : i - R.len0;
}

// ------------------------------------------------------------------------------------------
// Ring maintenance

__global__ void ring_zero_kernel(uint4* __restrict__ k, uint4* __restrict__ v, size_t n16) {
  const uint4 z = make_uint4(0u, 0u, 0u, 0u);
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride) {
    k[i] = z;
    v[i] = z;
  }
}

// Grid: x = batch * hkv rows of the ring, y = chunks of the source window.
__global__ void ring_fill_kernel(const int32_t* __restrict__ pos, const uint4* __restrict__ ks,
                                 const uint4* __restrict__ vs, uint4* __restrict__ kr,
                                 uint4* __restrict__ vr, int hkv, int src_len, int slots,
                                 int row16) {
  const int bg = blockIdx.x;
  const int t = pos[bg / hkv];
  if (t < 0) return;
  const size_t src_base = (size_t)bg * src_len * row16;
  const size_t dst_base = (size_t)bg * slots * row16;
  const int total = src_len * row16;
  for (int e = blockIdx.y * blockDim.x + threadIdx.x; e < total; e += gridDim.y * blockDim.x) {
    const int i = e / row16;
    const int c = e - i * row16;
    const long long s = (long long)t - src_len + i;  // absolute position of source row i
    if (s < 0) continue;
    const int slot = (int)(s % slots);
    kr[dst_base + (size_t)slot * row16 + c] = ks[src_base + (size_t)i * row16 + c];
    vr[dst_base + (size_t)slot * row16 + c] = vs[src_base + (size_t)i * row16 + c];
  }
}

// ------------------------------------------------------------------------------------------
// fp32 decode on vector ALUs.
//
// One workgroup (4 waves) per (sequence, KV head).  Each 16-lane quarter of a wave is a key
// stream: its lanes split head_dim (D/16 channels each), reduce the G dot products with
// lane shuffles and run its own online softmax over keys stream, stream + 16, ...; the 16
// stream states are merged with Eq.(lse) (Appendix A.4) at the end.
template <int D, int GMAX>
__global__ __launch_bounds__(256) void decode_f32_kernel(DecodeArgs a) {
  constexpr int E = D / 16;
  __shared__ float sm_acc[4][GMAX][D];
  __shared__ float sm_m[4][GMAX];
  __shared__ float sm_l[4][GMAX];

  const int bg = blockIdx.x;
  const int b = bg / a.hkv;
  const int g = bg - b * a.hkv;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int sub = lane & 15;
  const int stream = wave * 4 + (lane >> 4);
  const int G = a.group;
  float* out = (float*)a.out + ((size_t)b * a.hq + (size_t)g * G) * D;
  const int t = a.pos[b];
  if (t < 0) {
    for (int e = tid; e < G * D; e += 256) out[e] = 0.0f;
    if (a.pos_next != nullptr && g == 0 && tid == 0) a.pos_next[b] = t;
    return;
  }
  const Ranges R = ranges_for(a, t);
  if (a.pos_next != nullptr && g == 0 && tid == 0) a.pos_next[b] = t + 1;
  float* kring = (float*)a.k_ring + (size_t)bg * a.slots * D;
  float* vring = (float*)a.v_ring + (size_t)bg * a.slots * D;
  const float* knew = (const float*)a.k_new + (size_t)bg * D;
  const float* vnew = (const float*)a.v_new + (size_t)bg * D;

  // Fused append of the current token (slot t mod slots is outside the support).
  if (tid < D) {
    kring[(size_t)R.append_slot * D + tid] = knew[tid];
    vring[(size_t)R.append_slot * D + tid] = vnew[tid];
  }

  float qf[GMAX][E];
  const float* qrow = (const float*)a.q + ((size_t)b * a.hq + (size_t)g * G) * D + sub * E;
#pragma unroll
  for (int j = 0; j < GMAX; ++j)
#pragma unroll
    for (int e = 0; e < E; ++e) qf[j][e] = (j < G) ? qrow[(size_t)j * D + e] * a.scale_log2 : 0.0f;

  float m[GMAX], l[GMAX], acc[GMAX][E];
#pragma unroll
  for (int j = 0; j < GMAX; ++j) {
    m[j] = kNegInf;
    l[j] = 0.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) acc[j][e] = 0.0f;
  }

  const int n_total = R.n_ring + 1;
  for (int i = stream; i < n_total; i += 16) {
    const float* kp;
    const float* vp;
    if (i < R.n_ring) {
      const size_t off = (size_t)ring_slot(R, i) * D;
      kp = kring + off;
      vp = vring + off;
    } else {
      kp = knew;
      vp = vnew;
    }
    float kf[E], vf[E];
#pragma unroll
    for (int e = 0; e < E; e += 4) {
      const float4 k4 = *(const float4*)(kp + sub * E + e);
      const float4 v4 = *(const float4*)(vp + sub * E + e);
      kf[e] = k4.x; kf[e + 1] = k4.y; kf[e + 2] = k4.z; kf[e + 3] = k4.w;
      vf[e] = v4.x; vf[e + 1] = v4.y; vf[e + 2] = v4.z; vf[e + 3] = v4.w;
    }
#pragma unroll
    for (int j = 0; j < GMAX; ++j) {
      if (j < G) {
      float s = 0.0f;
#pragma unroll
      for (int e = 0; e < E; ++e) s = fmaf(qf[j][e], kf[e], s);
      s += __shfl_xor(s, 8, 16);
      s += __shfl_xor(s, 4, 16);
      s += __shfl_xor(s, 2, 16);
      s += __shfl_xor(s, 1, 16);
      const float mn = fmaxf(m[j], s);
      const float alpha = fast_exp2(m[j] - mn);  // m = -inf gives 0
      const float p = fast_exp2(s - mn);
      l[j] = l[j] * alpha + p;
#pragma unroll
      for (int e = 0; e < E; ++e) acc[j][e] = fmaf(p, vf[e], acc[j][e] * alpha);
      m[j] = mn;
      }
    }
  }

  // Merge the four streams of this wave (Eq.(lse)); empty streams carry m = -inf, l = 0.
#pragma unroll
  for (int off = 16; off <= 32; off <<= 1) {
#pragma unroll
    for (int j = 0; j < GMAX; ++j) {
      if (j < G) {
      const float mo = __shfl_xor(m[j], off);
      const float lo = __shfl_xor(l[j], off);
      const float mn = fmaxf(m[j], mo);
      const float a1 = (m[j] == kNegInf) ? 0.0f : fast_exp2(m[j] - mn);
      const float a2 = (mo == kNegInf) ? 0.0f : fast_exp2(mo - mn);
      l[j] = l[j] * a1 + lo * a2;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const float ao = __shfl_xor(acc[j][e], off);
        acc[j][e] = acc[j][e] * a1 + ao * a2;
      }
      m[j] = mn;
      }
    }
  }
  if (lane < 16) {
#pragma unroll
    for (int j = 0; j < GMAX; ++j) {
      if (j < G) {
#pragma unroll
        for (int e = 0; e < E; ++e) sm_acc[wave][j][sub * E + e] = acc[j][e];
        if (lane == 0) {
          sm_m[wave][j] = m[j];
          sm_l[wave][j] = l[j];
        }
      }
    }
  }
  __syncthreads();
  for (int idx = tid; idx < G * D; idx += 256) {
    const int j = idx / D;
    const int c = idx - j * D;
    float M = kNegInf;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, sm_m[w][j]);
    float L = 0.0f, O = 0.0f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float mw = sm_m[w][j];
      const float wt = (mw == kNegInf) ? 0.0f : fast_exp2(mw - M);
      L += wt * sm_l[w][j];
      O += wt * sm_acc[w][j][c];
    }
    out[idx] = O / L;
  }
}

// ------------------------------------------------------------------------------------------
// bf16 decode on matrix cores.
//
// One workgroup of NW waves per (sequence, KV head); wave w handles 32-key steps
// w, w + NW, ... of the unit's key list (ring keys, then the current token).  Per step:
//   scores  S^T[16 keys][16 heads] = K Q^T with v_mfma_f32_16x16x32_bf16, two tiles; the A
//           operand (lane l: key l%16, channels 32kk + 8(l/16) .. +7) is one 16-byte LDS read,
//           the B operand holds the group's queries, padded to 16 heads with zeros.
//   softmax lane (head h = l%16, quarter j = l/16) holds the scores of keys 4j..4j+3 and
//           16+4j..16+4j+3; the running maximum is shared across the four quarters.
//   values  O^T[16 channels][16 heads] += V^T P^T.  P^T's B operand is exactly the score
//           registers (rounded to bf16), so the key order of the contraction is fixed by the
//           score layout; V is read back from LDS transposed, one bf16 per lane and row.
// K and V rows travel from HBM straight into wave-private LDS tiles (global_load_lds_dwordx4
// with the non-temporal hint: the ring is read once per step), two steps deep: while step s
// computes, the loads of step s + NW are in flight, and step s + 2NW is issued right after.
// No loaded value lands in a register, so the only memory wait is the explicit
// vmcnt(OPS) at the top of a step: loads retire in issue order and exactly OPS loads (the
// next step's) are issued after the current step's.  Steps past the end are still issued,
// with every key reading the current token's cached row, to keep that count fixed.  Padded
// heads (h >= G) compute on zero queries and are never stored.  Wave results are merged
// through LDS with Eq.(lse) (Appendix A.4) and written as bf16 (RNE).
//
// Tile layouts.  One 16-byte DMA of the wave writes 1 KiB: lane l lands at byte 16 l, i.e.
// RPI whole rows.  K rows are contiguous; the 16-byte piece p of row r sits at piece slot
// p ^ kswz(r), which spreads the 16 rows read by one MFMA operand over all banks.  V groups of
// RPI rows are padded (and, for D = 64, the upper row quad is piece-swizzled) so that the
// transposed reads of rows 4j+e (j = 0..3) hit 32 distinct banks.
template <int D, int NW, bool NT, bool ROPE>
__global__ __launch_bounds__(NW * 64) void decode_bf16_kernel(DecodeArgs a) {
  // NT: stream the ring with the non-temporal hint (rings far larger than the caches); without
  // it, small rings that are re-read every step can stay cache-resident.
  constexpr int kPolicy = NT ? kCachePolicyNT : 0;
  constexpr int KK = D / 32;            // 32-channel slices of the score contraction
  constexpr int NB = D / 16;            // 16-channel blocks of the output
  constexpr int ROWB = D * 2;           // bytes of one K or V row
  constexpr int PPR = D / 8;            // 16-byte pieces per row
  constexpr int RPI = 64 / PPR;         // rows per 1 KiB DMA group
  constexpr int NG = 32 / RPI;          // DMA groups per step and tensor
  constexpr int VPITCH = 1024 + (D == 128 ? 32 : 64);
  constexpr int KTILE = 32 * ROWB;
  constexpr int VTILE = NG * VPITCH;
  constexpr int BUF = KTILE + VTILE;    // one step: K tile then V tile
  constexpr int OPS = 2 * NG;           // DMA instructions per step
  constexpr int QTILE = 16 * ROWB;      // the group's queries, 16 rows (heads >= G unused)
  constexpr int STAGE_BYTES = NW * (2 * BUF + QTILE);
  constexpr int MERGE_BYTES = NW * 16 * (D + 2) * 4;
  constexpr int SMEM = STAGE_BYTES > MERGE_BYTES ? STAGE_BYTES : MERGE_BYTES;
  __shared__ __align__(16) unsigned char smem[SMEM];

  const int bg = blockIdx.x;
  const int b = bg / a.hkv;
  const int g = bg - b * a.hkv;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int c16 = lane & 15;
  const int j4 = lane >> 4;
  const int G = a.group;
  uint16_t* out = (uint16_t*)a.out + ((size_t)b * a.hq + (size_t)g * G) * D;
  const int t = a.pos[b];
  if (t < 0) {
    for (int e = tid; e < G * D; e += NW * 64) out[e] = 0;
    if (a.pos_next != nullptr && g == 0 && tid == 0) a.pos_next[b] = t;
    return;
  }
  const Ranges R = ranges_for(a, t);
  const int n_total = R.n_ring + 1;
  uint16_t* kring = (uint16_t*)a.k_ring + (size_t)bg * a.slots * D;
  uint16_t* vring = (uint16_t*)a.v_ring + (size_t)bg * a.slots * D;
  const uint16_t* knew = (const uint16_t*)a.k_new + (size_t)bg * D;
  const uint16_t* vnew = (const uint16_t*)a.v_new + (size_t)bg * D;
  if (a.pos_next != nullptr && g == 0 && tid == 0) a.pos_next[b] = t + 1;

  // The current token's row for the append: loaded now, stored at the end, so that only the
  // store sits on the tail of a latency-bound launch.
  const bool appender = wave == 0 && lane < 2 * PPR;
  u32x4 append_row = {0u, 0u, 0u, 0u};
  if (appender)
    append_row = *(const u32x4*)((lane < PPR ? knew : vnew) + (lane % PPR) * 8);

  bf16x8 qB[KK];
  float m = kNegInf;
  float lsum = 0.0f;
  f32x4 acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  unsigned char* buf[2] = {smem + (wave * 2) * BUF, smem + (wave * 2 + 1) * BUF};
  unsigned char* qtile = smem + NW * 2 * BUF + wave * QTILE;
  const int nsteps = (n_total + 31) >> 5;

  // Rotary mode: queries and the new key are turned by position t inside this launch.  Their
  // raw values and the per-channel turn rates are loaded into registers here, before any K/V
  // load, so that the first step's vmcnt wait covers them; lanes l < PPR/2 hold the new key's
  // pieces l and l + PPR/2 (channels 8l.. and d/2 + 8l..), which pair up under the rotation.
  u32x4 qraw[ROPE ? KK : 1];
  u32x4 krot_lo = {0u, 0u, 0u, 0u}, krot_hi = {0u, 0u, 0u, 0u};
  double qturn[ROPE ? 4 * KK : 1], kturn[8];
  if constexpr (ROPE) {
    const uint16_t* qrow = (const uint16_t*)a.q + ((size_t)b * a.hq + (size_t)g * G +
                                                   (size_t)(c16 < G ? c16 : G - 1)) * D;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) qraw[kk] = *(const u32x4*)(qrow + 32 * kk + 8 * j4);
#pragma unroll
    for (int kk = 0; kk < KK / 2; ++kk)
#pragma unroll
      for (int e = 0; e < 8; ++e) qturn[kk * 8 + e] = a.rope_turns[32 * kk + 8 * j4 + e];
    const int kl = lane < PPR / 2 ? lane : 0;
    krot_lo = *(const u32x4*)(knew + kl * 8);
    krot_hi = *(const u32x4*)(knew + D / 2 + kl * 8);
#pragma unroll
    for (int e = 0; e < 8; ++e) kturn[e] = a.rope_turns[8 * kl + e];
  }

  // The group's query rows go to the wave's LDS query tile by the same DMA as K and V, ahead
  // of the first K/V loads, so the first step's vmcnt wait covers them too (rows of heads
  // >= G repeat head G-1 and are zeroed when read).
  if constexpr (!ROPE) {
    const uint16_t* qbase = (const uint16_t*)a.q + ((size_t)b * a.hq + (size_t)g * G) * D;
#pragma unroll
    for (int x = 0; x < 16 / RPI; ++x) {
      const int h = x * RPI + lane / PPR;
      const uint16_t* src = qbase + (size_t)(h < G ? h : G - 1) * D + (lane % PPR) * 8;
      __builtin_amdgcn_global_load_lds((const void*)src,
                                       (__attribute__((address_space(3))) void*)(qtile + x * 1024),
                                       16, 0, 0);
    }
  }

  // Row offset (elements) of key i in its ring, or of the current token's row.
  auto row_of = [&](int i, const uint16_t* ring, const uint16_t* fresh) -> const uint16_t* {
    return i < R.n_ring ? ring + (size_t)ring_slot(R, i) * D : fresh;
  };
  auto kswz = [](int r) -> int { return D == 128 ? (r & 15) : ((r >> 1) & 7); };
  auto vswz = [](int rr) -> int { return (D == 64 && rr >= 4) ? 2 : 0; };

  auto issue = [&](unsigned char* tile, int step) {
    const int k0 = step * 32;
    const int rr = lane / PPR;
    const int slot = lane % PPR;
#pragma unroll
    for (int x = 0; x < NG; ++x) {
      const int row = x * RPI + rr;
      const uint16_t* src = row_of(k0 + row, kring, knew) + (slot ^ kswz(row)) * 8;
      __builtin_amdgcn_global_load_lds((const void*)src,
                                       (__attribute__((address_space(3))) void*)(tile + x * 1024),
                                       16, 0, kPolicy);
    }
#pragma unroll
    for (int x = 0; x < NG; ++x) {
      const int row = x * RPI + rr;
      const uint16_t* src = row_of(k0 + row, vring, vnew) + (slot ^ vswz(rr)) * 8;
      __builtin_amdgcn_global_load_lds(
          (const void*)src, (__attribute__((address_space(3))) void*)(tile + KTILE + x * VPITCH),
          16, 0, kPolicy);
    }
  };

  auto compute = [&](const unsigned char* tile, int step) {
    // This step's tiles have landed once at most the next step's OPS loads are outstanding.
    __builtin_amdgcn_s_waitcnt(0x0F70 | (OPS & 15) | ((OPS >> 4) << 14));
    if constexpr (ROPE) {
      // The current token's K row arrived unrotated from k_new: overwrite it with the turned
      // key before the tile is read.
      if (step == (R.n_ring >> 5)) {
        const int rc = R.n_ring & 31;
        if (lane < PPR / 2) {
          unsigned char* row = (unsigned char*)tile + rc * ROWB;
          *(u32x4*)(row + ((lane ^ kswz(rc)) << 4)) = krot_lo;
          *(u32x4*)(row + (((lane + PPR / 2) ^ kswz(rc)) << 4)) = krot_hi;
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      }
    }
    const int k0 = step * 32;
    f32x4 s0 = {0.0f, 0.0f, 0.0f, 0.0f};
    f32x4 s1 = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const int p = 4 * kk + j4;
      const bf16x8 ka = *(const bf16x8*)(tile + c16 * ROWB + ((p ^ kswz(c16)) << 4));
      const bf16x8 kb = *(const bf16x8*)(tile + (16 + c16) * ROWB + ((p ^ kswz(16 + c16)) << 4));
      s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qB[kk], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kb, qB[kk], s1, 0, 0, 0);
    }
    float z[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      z[e] = s0[e] * a.scale_log2;
      z[4 + e] = s1[e] * a.scale_log2;
    }
    float mx = kNegInf;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int key = k0 + (e < 4 ? 4 * j4 + e : 16 + 4 * j4 + (e - 4));
      if (key >= n_total) z[e] = kNegInf;
      mx = fmaxf(mx, z[e]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mn = fmaxf(m, mx);
    const float alpha = fast_exp2(m - mn);  // 0 on the first step (m = -inf)
    float ps = 0.0f;
    bf16x8 pB;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float p = fast_exp2(z[e] - mn);
      ps += p;
      pB[e] = (__bf16)p;
    }
    lsum = lsum * alpha + ps;
    m = mn;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] *= alpha;
    const unsigned char* vt = tile + KTILE;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int col = 16 * nb + c16;
      bf16x8 va;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int row = e < 4 ? 4 * j4 + e : 16 + 4 * j4 + (e - 4);
        const int rr = row % RPI;
        const int off = (row / RPI) * VPITCH + rr * ROWB + (((col >> 3) ^ vswz(rr)) << 4) +
                        ((col & 7) << 1);
        va[e] = *(const __bf16*)(vt + off);
      }
      acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pB, acc[nb], 0, 0, 0);
    }
  };

  // Two-deep software pipeline with a uniform trip count (pairs of steps), then the odd one.
  const int my_steps = wave < nsteps ? (nsteps - wave + NW - 1) / NW : 0;
  int step = wave;
  issue(buf[0], step);
  issue(buf[1], step + NW);
  // Queries: wait until at most the two prefetched steps are outstanding, then read the
  // B operand (channels 32kk + 8j .. +7 of head c16; zero for padded heads).
  __builtin_amdgcn_s_waitcnt(0x0F70 | ((2 * OPS) & 15) | (((2 * OPS) >> 4) << 14));
  if constexpr (ROPE) {
    // Turn the queries (channel 32kk + 8j + e pairs with the same channel of slice kk + KK/2)
    // and the new key; round to bf16 as the matrix-core operands and the ring hold them.
    const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int kk = 0; kk < KK / 2; ++kk) {
      bf16x8 x = __builtin_bit_cast(bf16x8, qraw[kk]);
      bf16x8 y = __builtin_bit_cast(bf16x8, qraw[kk + KK / 2]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float cs, sn, ox, oy;
        rope_cos_sin(t, qturn[kk * 8 + e], cs, sn);
        rope_turn((float)x[e], (float)y[e], cs, sn, ox, oy);
        x[e] = (__bf16)ox;
        y[e] = (__bf16)oy;
      }
      qB[kk] = c16 < G ? x : __builtin_bit_cast(bf16x8, zero);
      qB[kk + KK / 2] = c16 < G ? y : __builtin_bit_cast(bf16x8, zero);
    }
    bf16x8 x = __builtin_bit_cast(bf16x8, krot_lo);
    bf16x8 y = __builtin_bit_cast(bf16x8, krot_hi);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float cs, sn, ox, oy;
      rope_cos_sin(t, kturn[e], cs, sn);
      rope_turn((float)x[e], (float)y[e], cs, sn, ox, oy);
      x[e] = (__bf16)ox;
      y[e] = (__bf16)oy;
    }
    krot_lo = __builtin_bit_cast(u32x4, x);
    krot_hi = __builtin_bit_cast(u32x4, y);
  }
#pragma unroll
  for (int kk = 0; kk < (ROPE ? 0 : KK); ++kk) {
    const u32x4 zero = {0u, 0u, 0u, 0u};
    const u32x4 w = *(const u32x4*)(qtile + c16 * ROWB + (4 * kk + j4) * 16);
    qB[kk] = __builtin_bit_cast(bf16x8, c16 < G ? w : zero);
  }
  for (int pair = 0; pair < my_steps / 2; ++pair) {
    __builtin_amdgcn_sched_barrier(0);
    compute(buf[0], step);
    __builtin_amdgcn_sched_barrier(0);
    issue(buf[0], step + 2 * NW);
    step += NW;
    __builtin_amdgcn_sched_barrier(0);
    compute(buf[1], step);
    __builtin_amdgcn_sched_barrier(0);
    issue(buf[1], step + 2 * NW);
    step += NW;
  }
  if (my_steps & 1) {
    __builtin_amdgcn_sched_barrier(0);
    compute(buf[0], step);
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);  // drain the trailing prefetches before LDS is reused

  // l per head: sum the four quarters' partial sums.
  lsum += __shfl_xor(lsum, 16);
  lsum += __shfl_xor(lsum, 32);

  __syncthreads();  // every wave is done with its tiles: reuse LDS for the merge
  float* sm_acc = (float*)smem;              // [NW][16 heads][D]
  float* sm_m = sm_acc + NW * 16 * D;         // [NW][16]
  float* sm_l = sm_m + NW * 16;               // [NW][16]
  if (c16 < G) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) sm_acc[(wave * 16 + c16) * D + 16 * nb + 4 * j4 + i] = acc[nb][i];
    if (j4 == 0) {
      sm_m[wave * 16 + c16] = m;
      sm_l[wave * 16 + c16] = lsum;
    }
  }
  __syncthreads();
  for (int idx = tid; idx < G * D; idx += NW * 64) {
    const int h = idx / D;
    const int c = idx - h * D;
    float M = kNegInf;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, sm_m[w * 16 + h]);
    float L = 0.0f, O = 0.0f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float mw = sm_m[w * 16 + h];
      const float wt = (mw == kNegInf) ? 0.0f : fast_exp2(mw - M);
      L += wt * sm_l[w * 16 + h];
      O += wt * sm_acc[(w * 16 + h) * D + c];
    }
    out[idx] = float_to_bf16_rne(O / L);
  }

  // Fused append of the current token.  Slot t mod slots holds a position outside the support
  // of t (and of every later step), so no read of this launch can observe the write.
  if constexpr (ROPE) {
    if (wave == 0 && lane < PPR / 2) {
      uint16_t* dst = kring + (size_t)R.append_slot * D;
      *(u32x4*)(dst + lane * 8) = krot_lo;
      *(u32x4*)(dst + D / 2 + lane * 8) = krot_hi;
    }
    if (appender && lane >= PPR)
      *(u32x4*)(vring + (size_t)R.append_slot * D + (lane % PPR) * 8) = append_row;
  } else if (appender) {
    *(u32x4*)((lane < PPR ? kring : vring) + (size_t)R.append_slot * D + (lane % PPR) * 8) =
        append_row;
  }
}

}  // namespace

// ------------------------------------------------------------------------------------------
// Launchers

hipError_t launch_ring_zero(void* k_ring, void* v_ring, size_t bytes, hipStream_t stream) {
  const size_t n16 = bytes / 16;
  size_t blocks = (n16 + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks == 0) blocks = 1;
  hipLaunchKernelGGL(ring_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                     (uint4*)k_ring, (uint4*)v_ring, n16);
  return hipGetLastError();
}

hipError_t launch_ring_fill(const int32_t* pos, const void* k_src, const void* v_src,
                            void* k_ring, void* v_ring, int32_t batch, int32_t hkv,
                            int32_t src_len, int32_t slots, int32_t row_bytes,
                            hipStream_t stream) {
  if (src_len == 0) return hipSuccess;
  const int row16 = row_bytes / 16;
  const int total = src_len * row16;
  int chunks = (total + 255) / 256;
  if (chunks > 64) chunks = 64;
  hipLaunchKernelGGL(ring_fill_kernel, dim3((unsigned)(batch * hkv), (unsigned)chunks), dim3(256),
                     0, stream, pos, (const uint4*)k_src, (const uint4*)v_src, (uint4*)k_ring,
                     (uint4*)v_ring, hkv, src_len, slots, row16);
  return hipGetLastError();
}

template <int D, int NW>
void launch_bf16_policy(const DecodeArgs& a, bool nt, hipStream_t stream) {
  const dim3 grid((unsigned)(a.batch * a.hkv));
  const dim3 block(NW * 64);
  if (a.rope) {
    if (nt) hipLaunchKernelGGL((decode_bf16_kernel<D, NW, true, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((decode_bf16_kernel<D, NW, false, true>), grid, block, 0, stream, a);
  } else {
    if (nt) hipLaunchKernelGGL((decode_bf16_kernel<D, NW, true, false>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((decode_bf16_kernel<D, NW, false, false>), grid, block, 0, stream, a);
  }
}

hipError_t launch_decode_bf16(const DecodeArgs& a, int32_t head_dim, hipStream_t stream) {
  // Workgroup width: long supports (up to >= 2048 keys) stream best with 4 waves per unit and
  // one workgroup per CU; so do launches with fewer units than CUs, where the latency of a
  // unit is what counts.  Otherwise 2 waves and two workgroups per CU.
  const int max_keys = a.mode == kSupportPBB ? a.block : a.window;
  const int units = a.batch * a.hkv;
  const bool wide = max_keys >= 2048 || units < 256;
  // Non-temporal loads once both rings exceed the 256 MiB last-level cache of the chip.
  const double ring_bytes = 4.0 * (double)units * (double)a.slots * (double)head_dim;
  const bool nt = ring_bytes > 256.0 * 1024.0 * 1024.0;
  if (head_dim == 128) {
    if (wide) launch_bf16_policy<128, 4>(a, nt, stream);
    else launch_bf16_policy<128, 2>(a, nt, stream);
  } else {
    if (wide) launch_bf16_policy<64, 4>(a, nt, stream);
    else launch_bf16_policy<64, 2>(a, nt, stream);
  }
  return hipGetLastError();
}

hipError_t launch_decode_f32(const DecodeArgs& a, int32_t head_dim, hipStream_t stream) {
  const dim3 grid((unsigned)(a.batch * a.hkv));
  const dim3 block(256);
  if (head_dim == 128) {
    if (a.group <= 4)
      hipLaunchKernelGGL((decode_f32_kernel<128, 4>), grid, block, 0, stream, a);
    else if (a.group <= 8)
      hipLaunchKernelGGL((decode_f32_kernel<128, 8>), grid, block, 0, stream, a);
    else
      hipLaunchKernelGGL((decode_f32_kernel<128, 16>), grid, block, 0, stream, a);
  } else {
    if (a.group <= 4)
      hipLaunchKernelGGL((decode_f32_kernel<64, 4>), grid, block, 0, stream, a);
    else if (a.group <= 8)
      hipLaunchKernelGGL((decode_f32_kernel<64, 8>), grid, block, 0, stream, a);
    else
      hipLaunchKernelGGL((decode_f32_kernel<64, 16>), grid, block, 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace pbb
