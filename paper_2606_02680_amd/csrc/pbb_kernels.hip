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
#include <mutex>
#include <type_traits>
#include <stdint.h>

#include "pbb_device.h"
#include "pbb_internal.h"

// Decode workspace of the allocation-free entry point (pbb_decode_step_noalloc): the unit
// counters and partial states of split launches, one copy per device, held until the process
// ends.  Host code never uses this name as an address: noalloc_scratch() below resolves the
// device address once per device and every kernel argument uses that.
static __device__ __align__(256) unsigned char scratch[pbb::kNoAllocScratchBytes];

namespace pbb {
namespace {

__global__ void scratch_clear_kernel(uint4* __restrict__ p, size_t n16) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n16) p[i] = make_uint4(0u, 0u, 0u, 0u);
}

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
// fp32 decode on matrix cores (v_mfma_f32_16x16x4_f32: fp32 operands and accumulation).
//
// One workgroup of NW waves per (sequence, KV head); wave w handles 16-key tiles w, w + NW, ...
// of the unit's key list (ring keys, then the current token).  Rows travel from memory straight
// into registers as matrix-core operands, the next tile's loads in flight while the current tile
// computes.  Lane l works in quarter j = l / 16 on row l % 16 of each 16 x 16 tile:
//   scores  S^T[16 keys][16 heads] = K Q^T in D/4 MFMAs; MFMA m contracts channel
//           16 (m / 4) + 4 j + m mod 4 in quarter j, so lane (key l%16, j) reads channels
//           16 x + 4 j .. +3 of its key row (x < D/16): each 16-byte load of the wave then
//           takes 64 contiguous bytes of each of 16 rows.  The B operand holds the queries
//           under the same map (scaled by scale * log2 e, zero for heads past G).  The result
//           gives lane (head l%16, j) keys 4j..4j+3 of the tile.
//   softmax column maxima across the quarters by permlane swaps; the reference moves only when
//           a column's maximum exceeds it by more than 8 (log2 units), decided wave-uniformly.
//   values  O^T += V^T P^T in D/4 MFMAs: row r of output tile nb is channel
//           64 (nb / 4) + 4 r + nb mod 4 and MFMA (nb, m) contracts key 4j + m in quarter j, so
//           the B operand is the lane's own weight of key 4j + m and lane (r, j) reads channels
//           64 y + 4 r .. +3 (y < D/64) of each of its four key rows: each 16-byte load of the
//           wave takes 256 contiguous bytes of each of 4 rows.
// Waves merge through LDS with Eq.(lse) (Appendix A.4); the append of the current token is
// done last (its slot is never read in the launch).
// Groups from this size on take the matrix-core fp32 kernel (a single query head per KV head
// streams as fast on the vector ALUs).
constexpr int kF32MatrixMinGroup = 2;

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2)))
void decode_f32_mfma_kernel(DecodeArgs a) {
  constexpr int KM = D / 4;     // MFMAs per score tile (channels per quarter)
  constexpr int E = D / 16;     // output tiles; channels per lane per key row of V
  constexpr int KQ = KM / 4;    // float4 loads of a lane's K channels
  constexpr int VQ = E / 4;     // float4 loads per V row
  typedef float f4 __attribute__((ext_vector_type(4)));
  __shared__ float sm_acc[NW][16][D];
  __shared__ float sm_m[NW][16];
  __shared__ float sm_l[NW][16];

  const int bg = blockIdx.x;
  const int b = bg / a.hkv;
  const int g = bg - b * a.hkv;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c16 = lane & 15;
  const int j4 = lane >> 4;
  const int G = a.group;
  float* out = (float*)a.out + ((size_t)b * a.hq + (size_t)g * G) * D;
  const int t = a.pos[b];
  if (t < 0) {
    for (int e = tid; e < G * D; e += NW * 64) out[e] = 0.0f;
    if (a.pos_next != nullptr && g == 0 && tid == 0) a.pos_next[b] = t;
    return;
  }
  const Ranges R = ranges_for(a, t);
  if (a.pos_next != nullptr && g == 0 && tid == 0) a.pos_next[b] = t + 1;
  float* kring = (float*)a.k_ring + (size_t)bg * a.slots * D;
  float* vring = (float*)a.v_ring + (size_t)bg * a.slots * D;
  const float* knew = (const float*)a.k_new + (size_t)bg * D;
  const float* vnew = (const float*)a.v_new + (size_t)bg * D;
  const int n_total = R.n_ring + 1;
  const int ntiles = (n_total + 15) >> 4;

  // Queries of head c16 (zero past G), channels (D/4) j4 + m, scaled into log2 units.
  float qf[KM];
  {
    const float* qrow = (const float*)a.q + ((size_t)b * a.hq + (size_t)g * G +
                                             (size_t)(c16 < G ? c16 : 0)) * D + 4 * j4;
#pragma unroll
    for (int m = 0; m < KM; ++m)
      qf[m] = c16 < G ? qrow[16 * (m >> 2) + (m & 3)] * a.scale_log2 : 0.0f;
  }
  // Row of key i of the unit: a ring slot, the current token, or (past the end) the current
  // token again, masked out of the softmax.
  auto krow = [&](int i) __attribute__((always_inline)) -> const float* {
    return i < R.n_ring ? kring + (size_t)ring_slot(R, i) * D : knew;
  };
  auto vrow = [&](int i) __attribute__((always_inline)) -> const float* {
    return i < R.n_ring ? vring + (size_t)ring_slot(R, i) * D : vnew;
  };
  auto load = [&](int tile, f4 (&kb)[KQ], f4 (&vb)[4][VQ]) __attribute__((always_inline)) {
    const int i0 = tile * 16;
    const float* kp = krow(i0 + c16) + 4 * j4;
#pragma unroll
    for (int q = 0; q < KQ; ++q) kb[q] = *(const f4*)(kp + 16 * q);
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const float* vp = vrow(i0 + 4 * j4 + m) + 4 * c16;
#pragma unroll
      for (int q = 0; q < VQ; ++q) vb[m][q] = *(const f4*)(vp + 64 * q);
    }
  };

  float mref = -1.0e30f;   // finite floor below any score: masked keys weigh exp2(-inf) = 0
  float lsum = 0.0f;
  f4 acc[E];
#pragma unroll
  for (int nb = 0; nb < E; ++nb) acc[nb] = f4{0.0f, 0.0f, 0.0f, 0.0f};

  auto compute = [&](int tile, const f4 (&kb)[KQ], const f4 (&vb)[4][VQ])
      __attribute__((always_inline)) {
    // Eight partial dot products (MFMAs m mod 8), summed pairwise: the matrix core adds each of
    // its four products into the accumulator with a rounding, so eight chains of D/8 sequential
    // products (instead of four of D/4) keep the scores' fp32 rounding at the level of a short
    // sum.
    f4 sp[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) sp[u] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int m = 0; m < KM; ++m)
      sp[m & 7] = __builtin_amdgcn_mfma_f32_16x16x4f32(kb[m >> 2][m & 3], qf[m], sp[m & 7], 0, 0, 0);
    f4 s = ((sp[0] + sp[1]) + (sp[2] + sp[3])) + ((sp[4] + sp[5]) + (sp[6] + sp[7]));
    const int i0 = tile * 16 + 4 * j4;
    float mx = kNegInf;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      s[e] = i0 + e < n_total ? s[e] : kNegInf;
      mx = fmaxf(mx, s[e]);
    }
    mx = max_xor16_32(mx);
    const bool grow = mx > mref + 8.0f;
    if (__builtin_amdgcn_ballot_w64(grow) != 0) {
      const float alpha = grow ? fast_exp2(mref - mx) : 1.0f;
      mref = grow ? mx : mref;
      lsum *= alpha;
#pragma unroll
      for (int nb = 0; nb < E; ++nb) acc[nb] *= alpha;
    }
    float p[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) p[e] = fast_exp2(s[e] - mref);
    lsum += (p[0] + p[1]) + (p[2] + p[3]);
    // The matrix core adds its four products into the accumulator one at a time, each with a
    // rounding, so the tile's 16 keys are first summed into a fresh partial (rounding on small
    // values) that then enters the running sum with a single addition: one rounding per tile
    // on the large sum instead of sixteen.  With the eight score chains above, the largest
    // output error over c4's shapes and tensors (G = 8, |o| up to ~18) drops from 1.4e-5 to
    // about 5e-6, against the 1e-5 bound.
#pragma unroll
    for (int nb = 0; nb < E; ++nb) {
      f4 part = __builtin_amdgcn_mfma_f32_16x16x4f32(vb[0][nb >> 2][nb & 3], p[0],
                                                    f4{0.0f, 0.0f, 0.0f, 0.0f}, 0, 0, 0);
#pragma unroll
      for (int m = 1; m < 4; ++m)
        part = __builtin_amdgcn_mfma_f32_16x16x4f32(vb[m][nb >> 2][nb & 3], p[m], part, 0, 0, 0);
      acc[nb] += part;
    }
  };

  f4 ka[KQ], kb2[KQ];
  f4 va[4][VQ], vb2[4][VQ];
  int tile = wave;
  if (tile < ntiles) load(tile, ka, va);
  while (tile < ntiles) {
    if (tile + NW < ntiles) load(tile + NW, kb2, vb2);
    compute(tile, ka, va);
    tile += NW;
    if (tile >= ntiles) break;
    if (tile + NW < ntiles) load(tile + NW, ka, va);
    compute(tile, kb2, vb2);
    tile += NW;
  }

  // Column sum over the four quarters; then the waves merge through LDS.
  lsum = sum_xor16_32(lsum);
  if (c16 < G) {
#pragma unroll
    for (int nb = 0; nb < E; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        sm_acc[wave][c16][64 * (nb >> 2) + 4 * (4 * j4 + i) + (nb & 3)] = acc[nb][i];
    if (j4 == 0) {
      sm_m[wave][c16] = mref;
      sm_l[wave][c16] = lsum;
    }
  }
  __syncthreads();
  for (int idx = tid; idx < G * D; idx += NW * 64) {
    const int h = idx / D;
    const int c = idx - h * D;
    float M = kNegInf;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, sm_m[w][h]);
    float L = 0.0f, O = 0.0f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float wt = fast_exp2(sm_m[w][h] - M);   // idle waves hold the floor: weight 0
      L += wt * sm_l[w][h];
      O += wt * sm_acc[w][h][c];
    }
    out[idx] = O / L;
  }

  // Fused append of the current token (slot t mod slots is outside the support).
  if (wave == 0 && lane < D / 4) {
    *(f4*)(kring + (size_t)R.append_slot * D + 4 * lane) = *(const f4*)(knew + 4 * lane);
    *(f4*)(vring + (size_t)R.append_slot * D + 4 * lane) = *(const f4*)(vnew + 4 * lane);
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
//           16+4j..16+4j+3.  A wave's first step sets the reference to the heads' maxima
//           (shared across the four quarters with permlane swaps); later steps compute no
//           maximum: the reference moves (and the accumulators are rescaled) only when some
//           lane's weights sum above 2^8, decided wave-uniformly, so weights stay <= 2^8 and
//           numerator and denominator share every reference (the same softmax).
//   values  O^T[16 channels][16 heads] += V^T P^T.  P^T's B operand is exactly the score
//           registers (rounded to bf16); V^T comes from transposed LDS reads
//           (ds_read_b64_tr_b16: lane i of each 16-lane group names 4 channels of key row
//           4j + i/4, lane c receives channel c of those four rows).
// K and V rows travel from HBM straight into wave-private LDS tiles (global_load_lds_dwordx4,
// with the non-temporal hint when the rings exceed the caches), two steps deep: while step s
// computes, the loads of step s + NW are in flight, and step s + 2NW is issued right after.
// A step's loads address the ring from a wave-uniform base: inside one slot range, row r of
// the step sits at a fixed per-lane offset from the range's first row; only steps that cross a
// range boundary, the current token or the end compute slots per lane.  The current token's row
// is not read from the ring: its K and V rows are loaded into registers at launch, and the wave
// that owns its step writes them into its LDS tiles (the DMA of that row, and of the padding
// after it, reads the support's first ring slot; the row is then overwritten).  No loaded value
// other than these lands in a register, so the only memory waits are the explicit vmcnt(OPS)
// at the top of a step: loads retire in issue order and exactly OPS loads (the next step's) are
// issued after the current step's.  Steps past the end are still issued (reading slot 0) to
// keep that count fixed.  Padded heads (h >= G) compute on zero queries and are never stored.
// Wave results are merged through LDS with Eq.(lse) (Appendix A.4), four channels per thread,
// and written as bf16 (RNE).
//
// Launch kinds.  The position is read through the scalar cache (no launch writes pos) after the
// queries and the current token's rows have been requested, so waiting for it does not wait for
// vector loads.  Whole-ring launches (WR: few units over rings of at most kWholeRingMaxSlots,
// where a step is latency-bound) issue the ring's 32-slot chunks, one per wave, before the
// position is known, and mask each chunk to the support afterwards: a 32-bit slot mask built
// from the two slot ranges sets the scores outside the support to -inf and zeroes their value
// operands in registers (slots never written may hold NaN bits); they append the current token
// as soon as the ring's loads have landed.  Split launches (SPLIT) spread a unit's steps over
// several workgroups that merge through the workspace (below).
//
// Tile layout.  One 16-byte DMA of the wave writes 1 KiB: lane l lands at byte 16 l, i.e. RPI
// whole rows.  Piece p of row r sits at piece slot p ^ swz(r), with swz(r) = 2 (r mod 8) for
// 256-byte rows and 2 ((r >> 1) mod 4) for 128-byte rows: both the 16-byte row reads of the
// scores and the transposed reads of the values hit distinct banks within every group of lanes
// that gfx950 serves per cycle.
// Device-coherent float store and load (agent scope): they bypass the caches that are not
// coherent across the chip's compute dies, without writing back or invalidating those caches.
//
// Ordering of the split merge.  The partial states are published and read ONLY through these
// agent-scope atomic accesses, and the unit counter is an agent-scope atomic add; the argument
// rests on how the AMDGPU backend's memory model for gfx942/gfx950 lowers them (LLVM
// AMDGPUUsage, "Memory Model GFX942"):
//   * an agent-scope atomic store or load is a global store/load with sc1 set: the store is
//     written through this die's L2 to the agent's coherence point, and the load is not served
//     from a stale line of a non-coherent cache;
//   * s_waitcnt vmcnt(0) returns only once every earlier store of the wave has been
//     acknowledged, i.e. is visible at that coherence point.  This is the completion step of
//     the backend's agent-scope release sequence; the other step of that sequence, the L2
//     write-back (buffer_wbl2 sc1), exists for stores made WITHOUT sc1, and no partial state is
//     written that way;
//   * the acquire sequence's L2 invalidation (buffer_inv sc1) likewise exists for later loads
//     made without sc1, and the merge reads the workspace only with sc1 loads, which it issues
//     after the counter's returned value has been observed (the flag goes through LDS and a
//     workgroup barrier, so no load can be performed before the add has returned).
// Hence: every store of a workgroup completes (vmcnt(0), then the barrier) before its count is
// added, and the last arriver's loads read the coherence point after the final count -- the
// guarantees a release add / acquire load pair would give, without the cache-wide write-back
// and invalidation (measured 3x slower, because the invalidation also evicts rings that stay
// cache-resident at small batch).  Relaxed accesses do not carry this guarantee in the
// language-level model; it is a property of the lowering above, and the graph-replay split
// tests exercise it every replay.
__device__ __forceinline__ void coherent_store(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float coherent_load(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int D, int NW, bool NT, bool ROPE, bool SPLIT, bool WR>
__global__ __launch_bounds__(NW * 64) void decode_bf16_kernel(DecodeArgs a) {
  static_assert(!(WR && SPLIT), "whole-ring launches are not split");
  constexpr int kPolicy = NT ? kCachePolicyNT : 0;
  constexpr int KK = D / 32;            // 32-channel slices of the score contraction
  constexpr int NB = D / 16;            // 16-channel blocks of the output
  constexpr int ROWB = D * 2;           // bytes of one K or V row
  constexpr int PPR = D / 8;            // 16-byte pieces per row
  constexpr int RPI = 64 / PPR;         // rows per 1 KiB DMA group
  constexpr int NG = 32 / RPI;          // DMA groups per step and tensor
  constexpr int TILE = 32 * ROWB;
  constexpr int BUF = 2 * TILE;         // one step: K tile then V tile
  constexpr int OPS = 2 * NG;           // DMA instructions per step
  // Step buffers per wave: two (a two-deep pipeline), or in whole-ring mode one per ring chunk
  // of the wave (chunks w, w + NW, ... of at most kWholeRingMaxSlots / 32).
  constexpr int CPW = WR ? (kWholeRingMaxSlots / 32 + NW - 1) / NW : 2;
  constexpr int NBUF = WR ? CPW : 2;
  constexpr int STAGE_BYTES = NW * NBUF * BUF;
  constexpr int MERGE_BYTES = NW * 16 * (D + 2) * 4;
  // Split launches merge up to kMaxSplitStates (splits x heads) states through LDS after the
  // wave merge area and the arrival flag.  Whole-ring launches keep the merge area after the
  // step buffers (no barrier before the partial states are written).
  constexpr int SPLIT_BYTES = SPLIT ? (2 * kMaxSplitStates + 16) * 4 : 0;
  constexpr int SMEM = WR ? STAGE_BYTES + MERGE_BYTES + 16
                          : (STAGE_BYTES > MERGE_BYTES + 16 + SPLIT_BYTES ? STAGE_BYTES
                                                                          : MERGE_BYTES + 16 + SPLIT_BYTES);
  __shared__ __align__(16) unsigned char smem[SMEM];

  const int S = SPLIT ? a.splits : 1;
  const int bg = blockIdx.x / S;        // unit: (sequence, KV head)
  const int sp = blockIdx.x - bg * S;   // this workgroup's share of the unit's steps
  const int b = bg / a.hkv;
  const int g = bg - b * a.hkv;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int c16 = lane & 15;
  const int j4 = lane >> 4;
  const int G = a.group;
  uint16_t* out = (uint16_t*)a.out + ((size_t)b * a.hq + (size_t)g * G) * D;
  uint16_t* kring = (uint16_t*)a.k_ring + (size_t)bg * a.slots * D;
  uint16_t* vring = (uint16_t*)a.v_ring + (size_t)bg * a.slots * D;
  const uint16_t* knew = (const uint16_t*)a.k_new + (size_t)bg * D;
  const uint16_t* vnew = (const uint16_t*)a.v_new + (size_t)bg * D;
  unsigned char* const wbuf = smem + wave * NBUF * BUF;   // this wave's step buffers

  auto swz = [](int r) -> int { return D == 128 ? 2 * (r & 7) : 2 * ((r >> 1) & 3); };

  // DMA of one step.  Lane l loads 16-byte piece (l mod PPR) ^ swz(row) of rows
  // row = x RPI + l / PPR, x < NG, into LDS byte x 1024 + 16 l of the K tile and of the V tile.
  const unsigned char* const kring_b = (const unsigned char*)kring;
  const unsigned char* const vring_b = (const unsigned char*)vring;
  uint32_t rowoff[NG];   // offset of this lane's piece of row x RPI + l / PPR from row 0
#pragma unroll
  for (int x = 0; x < NG; ++x) {
    const int row = x * RPI + lane / PPR;
    rowoff[x] = (uint32_t)(row * ROWB + (((lane % PPR) ^ swz(row)) << 4));
  }
  // Whole-ring mode (small rings, few units: latency-bound launches): wave w loads ring chunks
  // w, w + NW, ... (slots 32c .. 32c + 31, rows past the ring read its last slot) before the
  // position is known, so that the ring's loads and the position's load travel together; once
  // t is known, each chunk is masked to the support (the support always lies in the ring).
  const int nchunks = WR ? (a.slots + 31) >> 5 : 0;
  auto issue_chunk = [&](unsigned char* tile, int ch) {
    if (ch >= nchunks) return;
    const int s0 = ch * 32;
    uint32_t off[NG];
#pragma unroll
    for (int x = 0; x < NG; ++x) {
      const int row = x * RPI + lane / PPR;
      off[x] = s0 + 31 < a.slots ? (uint32_t)(s0 * ROWB) + rowoff[x]
                                 : (uint32_t)(min(s0 + row, a.slots - 1) * ROWB +
                                              (((lane % PPR) ^ swz(row)) << 4));
    }
#pragma unroll
    for (int x = 0; x < NG; ++x)
      __builtin_amdgcn_global_load_lds((const void*)(kring_b + off[x]),
                                       (__attribute__((address_space(3))) void*)(tile + x * 1024),
                                       16, 0, kPolicy);
#pragma unroll
    for (int x = 0; x < NG; ++x)
      __builtin_amdgcn_global_load_lds((const void*)(vring_b + off[x]),
                                       (__attribute__((address_space(3))) void*)(tile + TILE + x * 1024),
                                       16, 0, kPolicy);
  };
  if constexpr (WR)
    for (int c = 0; c < CPW; ++c) issue_chunk(wbuf + c * BUF, wave + c * NW);

  // The current token's K and V rows (lanes < PPR: K piece l, lanes PPR..2PPR-1: V piece l-PPR),
  // in every wave: the wave that owns the token's step writes them into its tiles, and wave 0
  // stores them into the ring at the end.
  const bool rowlane = lane < 2 * PPR;
  u32x4 cur_row = {0u, 0u, 0u, 0u};
  if (rowlane) cur_row = *(const u32x4*)((lane < PPR ? knew : vnew) + (lane % PPR) * 8);

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

  // The group's queries as the B operand (channels 32kk + 8j .. +7 of head c16), loaded into
  // registers ahead of the first K/V loads so that the first step's vmcnt wait covers them
  // (lanes of heads >= G load head G-1 and are zeroed when used).
  u32x4 qload[ROPE ? 1 : KK];
  if constexpr (!ROPE) {
    const uint16_t* qrow = (const uint16_t*)a.q + ((size_t)b * a.hq + (size_t)g * G +
                                                   (size_t)(c16 < G ? c16 : G - 1)) * D;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) qload[kk] = *(const u32x4*)(qrow + 32 * kk + 8 * j4);
  }

  // The position through the scalar cache (pos is never written during a launch: pos_next
  // may not alias it), so that waiting for it does not wait for the vector loads in flight.
  const int t = ((const __attribute__((address_space(4))) int32_t*)(const void*)a.pos)[b];
  if (t < 0) {
    if constexpr (WR) __builtin_amdgcn_s_waitcnt(0x0F70);   // no LDS load outlives the workgroup
    if (sp == 0)
      for (int e = tid; e < G * D; e += NW * 64) out[e] = 0;
    if (a.pos_next != nullptr && g == 0 && sp == 0 && tid == 0) a.pos_next[b] = t;
    return;
  }
  const Ranges R = ranges_for(a, t);
  const int n_total = R.n_ring + 1;
  const int pad_slot = R.n_ring > 0 ? ring_slot(R, 0) : 0;   // a slot the support reads
  if (a.pos_next != nullptr && g == 0 && sp == 0 && tid == 0) a.pos_next[b] = t + 1;
  // Whole-ring mode: slot s is read iff it lies in one of the support's two slot ranges or is
  // the current token's (which takes k_new / v_new).  Bit i of chunk_mask(ch): slot 32 ch + i
  // (wave-uniform; slots past the ring are never in a range).
  auto chunk_mask = [&](int ch) -> uint32_t {
    const int lo = ch * 32;
    auto bits = [&](int a0, int a1) -> uint32_t {   // slots [a0, a1) within the chunk
      const int x0 = max(a0, lo) - lo, x1 = min(a1, lo + 32) - lo;
      if (x1 <= x0) return 0u;
      return (x1 - x0 == 32 ? 0xFFFFFFFFu : ((1u << (x1 - x0)) - 1u)) << x0;
    };
    uint32_t mk = bits(R.base0, R.base0 + R.len0) | bits(0, R.n_ring - R.len0);
    const int ap = R.append_slot - lo;
    if (ap >= 0 && ap < 32) mk |= 1u << ap;
    return mk;
  };


  bf16x8 qB[KK];
  float m = kNegInf;
  float lsum = 0.0f;
  bool fresh = true;  // no step computed yet by this wave
  f32x4 acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  const int nsteps = (n_total + 31) >> 5;
  // Steps [st_lo, st_hi) of the unit belong to this workgroup.
  const int st_lo = SPLIT ? (int)(((long long)sp * nsteps) / S) : 0;
  const int st_hi = SPLIT ? (int)(((long long)(sp + 1) * nsteps) / S) : nsteps;
  // later rows are only read to keep the wait counts fixed
  const int k_lim = SPLIT ? st_hi * 32 : 0x7fffffff;

  auto issue = [&](unsigned char* tile, int step) {
    const int k0 = step * 32;
    auto dma = [&](const unsigned char* base, int x, uint32_t off, int vt) {
      __builtin_amdgcn_global_load_lds(
          (const void*)(base + off),
          (__attribute__((address_space(3))) void*)(tile + vt * TILE + x * 1024), 16, 0, kPolicy);
    };
    if (k0 < k_lim && (k0 + 31 < R.len0 || (k0 >= R.len0 && k0 + 31 < R.n_ring))) {
      // The whole step lies in one slot range: rows are consecutive slots.
      const int s0 = k0 < R.len0 ? R.base0 + k0 : k0 - R.len0;
      const size_t sh = (size_t)s0 * ROWB;
#pragma unroll
      for (int x = 0; x < NG; ++x) dma(kring_b + sh, x, rowoff[x], 0);
#pragma unroll
      for (int x = 0; x < NG; ++x) dma(vring_b + sh, x, rowoff[x], 1);
    } else {
      // Per-lane slots: range boundary, the current token and the padding after it (read from
      // the support's first ring slot, pad_slot: real data, whose weights are then 0; the
      // current token's row is replaced in LDS), or rows past this workgroup's steps (slot 0,
      // never used).
      uint32_t off[NG];
#pragma unroll
      for (int x = 0; x < NG; ++x) {
        const int row = x * RPI + lane / PPR;
        const int i = k0 + row;
        const int slot = k0 >= k_lim ? 0
                         : (i >= R.n_ring ? pad_slot : (i < R.len0 ? R.base0 + i : i - R.len0));
        off[x] = (uint32_t)(slot * ROWB + (((lane % PPR) ^ swz(row)) << 4));
      }
#pragma unroll
      for (int x = 0; x < NG; ++x) dma(kring_b, x, off[x], 0);
#pragma unroll
      for (int x = 0; x < NG; ++x) dma(vring_b, x, off[x], 1);
    }
  };

  // LDS read addresses (buffer 0 of this wave): K row operands (row c16, piece 4kk + j4; row
  // 16 + c16 a fixed distance on) and transposed V reads of chunk nb (row 4j + c16/4, channels
  // 16nb + 4(c16 mod 4) .. +3; rows 16.. a fixed distance on).
  uint32_t kaddr[KK], vaddr[NB];
  {
    const uint32_t base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)wbuf;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
      kaddr[kk] = base + c16 * ROWB + (((4 * kk + j4) ^ swz(c16)) << 4);
    const int r = 4 * j4 + (c16 >> 2);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      vaddr[nb] = base + TILE + r * ROWB + (((2 * nb + ((c16 & 3) >> 1)) ^ swz(r)) << 4) +
                  ((c16 & 1) << 3);
  }
  const __attribute__((address_space(3))) unsigned char* lds0 = nullptr;
  const float c = a.scale_log2;
  // the step (whole-ring mode: the chunk) that holds the current token, and its row there
  const int cur_step = WR ? (R.append_slot >> 5) : (R.n_ring >> 5);
  const int rc = WR ? (R.append_slot & 31) : (R.n_ring & 31);

  // bi selects a step buffer at compile time; bo (whole-ring mode) adds a run-time offset, so
  // that the chunks of one wave run through a single copy of this code.
  auto compute = [&](auto bi, int step, uint32_t bo) {
    constexpr uint32_t BO = decltype(bi)::value * BUF;
    // This step's tiles have landed once at most the next step's OPS loads are outstanding.
    __builtin_amdgcn_s_waitcnt(0x0F70 | (OPS & 15) | ((OPS >> 4) << 14));
    // Whole-ring mode: this lane's keys (4j4 + e and 16 + 4j4 + e, e < 4) that the support
    // reads, from the chunk's slot mask.
    uint32_t kbits = 0;
    if constexpr (WR) {
      const uint32_t cm = chunk_mask(step);
      kbits = ((cm >> (4 * j4)) & 0xFu) | (((cm >> (16 + 4 * j4)) & 0xFu) << 4);
    }
    if (step == cur_step) {
      // The current token's row arrived from pad_slot: overwrite it with k_new / v_new (the
      // turned key in rotary mode).  The rows after it (this step's padding) get weight 0; they
      // hold the support's first ring row, so 0 * V stays 0.  A support with no ring key
      // (t = 0) has no such row: its padding came from slot 0, which may hold bits that were
      // never written (0 * NaN would reach the output), so its V rows are zeroed.  Padded K
      // rows need nothing: their scores are replaced by -inf below.
      unsigned char* tile = wbuf + BO + bo;
      if (!WR && R.n_ring == 0) {
        const u32x4 zero = {0u, 0u, 0u, 0u};
        for (int e = lane; e < 31 * PPR; e += 64)
          *(u32x4*)(tile + TILE + (1 + e / PPR) * ROWB + (e % PPR) * 16) = zero;
      }
      if constexpr (ROPE) {
        if (lane < PPR / 2) {
          unsigned char* row = tile + rc * ROWB;
          *(u32x4*)(row + ((lane ^ swz(rc)) << 4)) = krot_lo;
          *(u32x4*)(row + (((lane + PPR / 2) ^ swz(rc)) << 4)) = krot_hi;
        }
        if (rowlane && lane >= PPR)
          *(u32x4*)(tile + TILE + rc * ROWB + (((lane - PPR) ^ swz(rc)) << 4)) = cur_row;
      } else if (rowlane) {
        *(u32x4*)(tile + (lane >= PPR ? TILE : 0) + rc * ROWB + (((lane % PPR) ^ swz(rc)) << 4)) =
            cur_row;
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    }
    const int k0 = step * 32;
    f32x4 s0 = {0.0f, 0.0f, 0.0f, 0.0f};
    f32x4 s1 = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const auto* p = lds0 + kaddr[kk] + BO + bo;
      const bf16x8 ka = *(const __attribute__((address_space(3))) bf16x8*)(p);
      const bf16x8 kb = *(const __attribute__((address_space(3))) bf16x8*)(p + 16 * ROWB);
      s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qB[kk], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kb, qB[kk], s1, 0, 0, 0);
    }
    // V^T reads go out now, under the softmax arithmetic.
    u32x2 vr[2 * NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      vr[2 * nb] = tr_read<BO>(vaddr[nb] + bo);
      vr[2 * nb + 1] = tr_read<BO + 16 * ROWB>(vaddr[nb] + bo);
    }
    if constexpr (WR) {
      // Slots outside the support do not count.
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if (!((kbits >> e) & 1u)) {
          if (e < 4) s0[e] = kNegInf;
          else s1[e - 4] = kNegInf;
        }
      }
    } else if (k0 + 32 > n_total) {
      // Keys past the current token (the last step's padding) do not count.
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int key = k0 + (e < 4 ? 4 * j4 + e : 16 + 4 * j4 + (e - 4));
        if (key >= n_total) {
          if (e < 4) s0[e] = kNegInf;
          else s1[e - 4] = kNegInf;
        }
      }
    }
    // Online softmax with a lazily moved reference m (Eq.(lse) rescaling): a wave's first step
    // sets m to its columns' maxima; later steps take their weights against m and move it (the
    // accumulators rescaled, the weights taken again) only when the eight weights of some lane
    // sum above 2^8 or to infinity -- whenever a score rises more than 8 log2 units above m,
    // and when several rise more than 5 -- so no other step computes a maximum.  Numerator and
    // denominator share every reference; the weights that enter them stay <= 2^8.
    auto move_reference = [&]() {
      float mx = fmaxf(fmaxf(fmaxf(s0[0], s0[1]), fmaxf(s0[2], s0[3])),
                       fmaxf(fmaxf(s1[0], s1[1]), fmaxf(s1[2], s1[3])));
      const float cand = max_xor16_32(mx) * c;
      const bool grow = cand > m;
      const float alpha = grow ? fast_exp2(m - cand) : 1.0f;   // 0 on the first step
      m = grow ? cand : m;
      lsum *= alpha;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[nb] *= alpha;
    };
    // The weights enter the value product rounded to bf16; the denominator sums the same
    // rounded weights, so the output is an exactly normalised average of the values under
    // those weights.  (Summing the unrounded weights instead leaves a mismatch of up to 2^-9
    // relative that scales with |o| itself, e.g. when one key carries almost all the weight.)
    float ps;
    bf16x8 pB;
    auto weights = [&]() {
      float sum = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float sc = e < 4 ? s0[e] : s1[e - 4];
        pB[e] = (__bf16)fast_exp2(__builtin_fmaf(sc, c, -m));
        sum += (float)pB[e];
      }
      ps = sum;
      return !(sum <= kWeightCap);
    };
    if (fresh) move_reference();
    fresh = false;
    if (__builtin_amdgcn_ballot_w64(weights()) != 0) {
      move_reference();
      weights();
    }
    lsum += ps;
    if constexpr (NB == 8) {
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(vr[0]), "+v"(vr[1]), "+v"(vr[2]), "+v"(vr[3]), "+v"(vr[4]),
                     "+v"(vr[5]), "+v"(vr[6]), "+v"(vr[7]), "+v"(vr[8]), "+v"(vr[9]),
                     "+v"(vr[10]), "+v"(vr[11]), "+v"(vr[12]), "+v"(vr[13]), "+v"(vr[14]),
                     "+v"(vr[15]));
    } else {
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(vr[0]), "+v"(vr[1]), "+v"(vr[2]), "+v"(vr[3]), "+v"(vr[4]),
                     "+v"(vr[5]), "+v"(vr[6]), "+v"(vr[7]));
    }
    if constexpr (WR) {
      // Values of slots outside the support are zeroed in registers: their weights are 0, but
      // the slots may hold bits that were never written (0 * NaN would reach the output).
      // Operand element e (bf16 half e mod 2 of dword e / 2) is key e of this lane.
      uint32_t vm[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        vm[i] = (((kbits >> (2 * i)) & 1u) ? 0x0000FFFFu : 0u) |
                (((kbits >> (2 * i + 1)) & 1u) ? 0xFFFF0000u : 0u);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        vr[2 * nb][0] &= vm[0];
        vr[2 * nb][1] &= vm[1];
        vr[2 * nb + 1][0] &= vm[2];
        vr[2 * nb + 1][1] &= vm[3];
      }
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const u32x4 w = {vr[2 * nb][0], vr[2 * nb][1], vr[2 * nb + 1][0], vr[2 * nb + 1][1]};
      acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, w), pB, acc[nb],
                                                        0, 0, 0);
    }
  };

  // Two-deep software pipeline with a uniform trip count (pairs of steps), then the odd one.
  const int my_steps = wave < st_hi - st_lo ? (st_hi - st_lo - wave + NW - 1) / NW : 0;
  int step = st_lo + wave;
  if constexpr (WR) {
    // queries, the current row and this wave's ring chunks have all landed
    __builtin_amdgcn_s_waitcnt(0x0F70);
  } else {
    issue(wbuf, step);
    issue(wbuf + BUF, step + NW);
    // Queries: wait until at most the two prefetched steps are outstanding (zero for padded
    // heads).
    __builtin_amdgcn_s_waitcnt(0x0F70 | ((2 * OPS) & 15) | (((2 * OPS) >> 4) << 14));
  }
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
    qB[kk] = __builtin_bit_cast(bf16x8, c16 < G ? qload[kk] : zero);
  }
  auto append_token = [&]() {
    // Fused append of the current token (by the unit's first workgroup).  Slot t mod slots
    // holds a position outside the support of t (and of every later step).
    if (wave == 0 && sp == 0) {
      if constexpr (ROPE) {
        if (lane < PPR / 2) {
          uint16_t* dst = kring + (size_t)R.append_slot * D;
          *(u32x4*)(dst + lane * 8) = krot_lo;
          *(u32x4*)(dst + D / 2 + lane * 8) = krot_hi;
        }
        if (rowlane && lane >= PPR)
          *(u32x4*)(vring + (size_t)R.append_slot * D + (lane % PPR) * 8) = cur_row;
      } else if (rowlane) {
        *(u32x4*)((lane < PPR ? kring : vring) + (size_t)R.append_slot * D + (lane % PPR) * 8) =
            cur_row;
      }
    }
  };
  // Whole-ring launches append right away: every ring load of the launch has completed, so the
  // store overlaps the computation instead of ending the launch.
  if constexpr (WR) append_token();
  if constexpr (WR) {
    // each wave computes its chunks that hold some slot of the support, one copy of the step
    // code in a loop
    for (int c = 0; c < CPW; ++c) {
      const int ch = wave + c * NW;
      if (ch < nchunks && chunk_mask(ch) != 0u) {
        __builtin_amdgcn_sched_barrier(0);
        compute(std::integral_constant<int, 0>{}, ch, (uint32_t)(c * BUF));
      }
    }
  }
  for (int pair = 0; pair < (WR ? 0 : my_steps / 2); ++pair) {
    __builtin_amdgcn_sched_barrier(0);
    compute(std::integral_constant<int, 0>{}, step, 0u);
    __builtin_amdgcn_sched_barrier(0);
    issue(wbuf, step + 2 * NW);
    step += NW;
    __builtin_amdgcn_sched_barrier(0);
    compute(std::integral_constant<int, 1>{}, step, 0u);
    __builtin_amdgcn_sched_barrier(0);
    issue(wbuf + BUF, step + 2 * NW);
    step += NW;
  }
  if (!WR && (my_steps & 1)) {
    __builtin_amdgcn_sched_barrier(0);
    compute(std::integral_constant<int, 0>{}, step, 0u);
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);  // drain the trailing prefetches before LDS is reused

  // l per head: sum the four quarters' partial sums.
  lsum = sum_xor16_32(lsum);

  if constexpr (!WR) __syncthreads();  // every wave is done with its tiles: reuse LDS for the merge
  float* sm_acc = (float*)(smem + (WR ? STAGE_BYTES : 0));   // [NW][16 heads][D]
  float* sm_m = sm_acc + NW * 16 * D;         // [NW][16]
  float* sm_l = sm_m + NW * 16;               // [NW][16]
  if (c16 < G) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      *(f32x4*)(sm_acc + (wave * 16 + c16) * D + 16 * nb + 4 * j4) = acc[nb];
    if (j4 == 0) {
      sm_m[wave * 16 + c16] = m;
      sm_l[wave * 16 + c16] = lsum;
    }
  }
  __syncthreads();
  // This workgroup's state per head: reference M (log2 units), sum L, unnormalised output O;
  // each thread takes 4 consecutive channels of one head.
  float* part = SPLIT ? a.ws_part + ((size_t)bg * S + sp) * G * (D + 2) : nullptr;
  constexpr int QD = D / 4;
  for (int i4 = tid; i4 < G * QD; i4 += NW * 64) {
    const int h = i4 / QD;
    const int q = i4 - h * QD;
    float mw[NW];
    float M = kNegInf;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      mw[w] = sm_m[w * 16 + h];
      M = fmaxf(M, mw[w]);
    }
    float L = 0.0f;
    f32x4 O = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float wt = (mw[w] == kNegInf) ? 0.0f : fast_exp2(mw[w] - M);
      L += wt * sm_l[w * 16 + h];
      const f32x4 o = *(const f32x4*)(sm_acc + (w * 16 + h) * D + 4 * q);
#pragma unroll
      for (int c4 = 0; c4 < 4; ++c4) O[c4] += wt * o[c4];
    }
    if constexpr (!SPLIT) {
      u32x2 w2;
      w2[0] = (uint32_t)float_to_bf16_rne(O[0] / L) | ((uint32_t)float_to_bf16_rne(O[1] / L) << 16);
      w2[1] = (uint32_t)float_to_bf16_rne(O[2] / L) | ((uint32_t)float_to_bf16_rne(O[3] / L) << 16);
      *(u32x2*)(out + h * D + 4 * q) = w2;
    } else {
#pragma unroll
      for (int c4 = 0; c4 < 4; ++c4) coherent_store(part + h * D + 4 * q + c4, O[c4]);
      if (q == 0) {
        coherent_store(part + G * D + h, M);
        coherent_store(part + G * D + G + h, L);
      }
    }
  }
  if constexpr (SPLIT) {
    // The last of the unit's workgroups to finish merges all S states (Eq.(lse)) and resets
    // the unit's counter for the next launch.  The states travel through device-coherent
    // stores and loads; every store of this workgroup has completed (the wait below, then the
    // barrier) before its count is added, so the workgroup that observes the final count
    // reads complete states.  No cache-wide write-back or invalidation is involved.
    int* last = (int*)(smem + MERGE_BYTES);
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this thread's stores have completed
    __syncthreads();
    if (tid == 0)
      *last = __hip_atomic_fetch_add(&a.counters[bg], 1u, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT) == (unsigned)(S - 1) ? 1 : 0;
    __syncthreads();
    if (*last) {
      // The S states' maxima and sums go to LDS first (all loads of a thread in flight
      // together), one thread per head turns them into weights exp2(m_s - M) and the total
      // L, and every output element then sums its S partial outputs, issuing several loads
      // before waiting: a handful of serial memory round trips instead of two per split and
      // element.
      const float* p0 = a.ws_part + (size_t)bg * S * G * (D + 2);
      float* wm = (float*)(smem + MERGE_BYTES + 16);   // [S][G] maxima, then weights
      float* wl = wm + S * G;                          // [S][G] sums
      float* hl = wl + S * G;                          // [G] totals
      for (int i = tid; i < S * G; i += NW * 64) {
        const int sx = i / G;
        const float* ps = p0 + (size_t)sx * G * (D + 2) + G * D + (i - sx * G);
        const float mv = coherent_load(ps);
        const float lv = coherent_load(ps + G);
        wm[i] = mv;
        wl[i] = lv;
      }
      __syncthreads();
      if (tid < G) {
        float M = kNegInf;
        for (int sx = 0; sx < S; ++sx) M = fmaxf(M, wm[sx * G + tid]);
        float L = 0.0f;
        for (int sx = 0; sx < S; ++sx) {
          const float ms = wm[sx * G + tid];
          const float wt = (ms == kNegInf) ? 0.0f : fast_exp2(ms - M);
          wm[sx * G + tid] = wt;
          L += wt * wl[sx * G + tid];
        }
        hl[tid] = L;
      }
      __syncthreads();
      for (int idx = tid; idx < G * D; idx += NW * 64) {
        const int h = idx / D;
        float O = 0.0f;
        for (int s0 = 0; s0 < S; s0 += 8) {
          // eight loads in flight per wait; past the last split the loads repeat it (in
          // bounds) and are not added
          float o[8];
#pragma unroll
          for (int j = 0; j < 8; ++j)
            o[j] = coherent_load(p0 + (size_t)min(s0 + j, S - 1) * G * (D + 2) + idx);
#pragma unroll
          for (int j = 0; j < 8; ++j)
            if (s0 + j < S) O += wm[(s0 + j) * G + h] * o[j];
        }
        out[idx] = float_to_bf16_rne(O / hl[h]);
      }
      if (tid == 0)
        __hip_atomic_store(&a.counters[bg], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }

  // Stepped launches append at the end: no read of this launch can observe the write (the slot
  // holds a position outside the support).
  if constexpr (!WR) append_token();
}

}  // namespace

// ------------------------------------------------------------------------------------------
// Launchers

hipError_t noalloc_scratch(void** ptr, hipStream_t stream) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    // The counter block must start at zero (every launch leaves it zero again); it is cleared
    // by a fill kernel, which a graph capture may record.
    hipLaunchKernelGGL(scratch_clear_kernel, dim3(1), dim3(64), 0, stream, (uint4*)p,
                       pbb::kCounterBytes / 16);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

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
  const dim3 grid((unsigned)(a.batch * a.hkv * a.splits));
  const dim3 block(NW * 64);
  if (a.splits > 1) {
    if (a.rope) {
      if (nt) hipLaunchKernelGGL((decode_bf16_kernel<D, NW, true, true, true, false>), grid, block, 0, stream, a);
      else hipLaunchKernelGGL((decode_bf16_kernel<D, NW, false, true, true, false>), grid, block, 0, stream, a);
    } else {
      if (nt) hipLaunchKernelGGL((decode_bf16_kernel<D, NW, true, false, true, false>), grid, block, 0, stream, a);
      else hipLaunchKernelGGL((decode_bf16_kernel<D, NW, false, false, true, false>), grid, block, 0, stream, a);
    }
    return;
  }
  if (a.rope) {
    if (nt) hipLaunchKernelGGL((decode_bf16_kernel<D, NW, true, true, false, false>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((decode_bf16_kernel<D, NW, false, true, false, false>), grid, block, 0, stream, a);
  } else {
    if (nt) hipLaunchKernelGGL((decode_bf16_kernel<D, NW, true, false, false, false>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((decode_bf16_kernel<D, NW, false, false, false, false>), grid, block, 0, stream, a);
  }
}

// Whole-ring launches: one workgroup of kWholeRingWaves waves per unit, rings of at most 256
// slots prefetched before the positions are read (cache-resident: no non-temporal hint).
template <int D>
void launch_bf16_whole(const DecodeArgs& a, hipStream_t stream) {
  constexpr int NW = kWholeRingWaves;
  const dim3 grid((unsigned)(a.batch * a.hkv)), block(NW * 64);
  if (a.rope) hipLaunchKernelGGL((decode_bf16_kernel<D, NW, false, true, false, true>), grid, block, 0, stream, a);
  else hipLaunchKernelGGL((decode_bf16_kernel<D, NW, false, false, false, true>), grid, block, 0, stream, a);
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
  // Latency-bound launches over small rings prefetch the whole ring with the positions.
  if (a.splits <= 1 && a.slots <= kWholeRingMaxSlots && units <= kWholeRingMaxUnits) {
    if (head_dim == 128) launch_bf16_whole<128>(a, stream);
    else launch_bf16_whole<64>(a, stream);
    return hipGetLastError();
  }
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
  if (a.group >= kF32MatrixMinGroup) {
    if (head_dim == 128)
      hipLaunchKernelGGL((decode_f32_mfma_kernel<128, 4>), grid, dim3(256), 0, stream, a);
    else
      hipLaunchKernelGGL((decode_f32_mfma_kernel<64, 4>), grid, dim3(256), 0, stream, a);
    return hipGetLastError();
  }
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
