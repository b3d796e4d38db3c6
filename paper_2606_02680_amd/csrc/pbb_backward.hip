// HIP backward of the PBB (and SWA) prefill attention on gfx950: gradients of q, k, v for
// training (the paper's fused kernel includes backward propagation, Sec. 3; its grouped backward
// sums the gradients of the query heads that share a KV head, Appendix F.4).
//
// For target t with support A(t), p_s = exp(z_s - lse_t), z_s = scale q_t.k_s (Eq.(attention);
// lse_t the forward's log-partition, Appendix A.4 Eq.(lse)) and upstream gradient g_t:
//   dv_s += p_s g_t
//   ds_s  = p_s (g_t.v_s - delta_t),   delta_t = g_t.o_t
//   dq_t  = scale sum_s ds_s k_s,      dk_s += scale ds_s q_t
// summed over the query heads of each KV head for dk and dv.  Two launches:
//   dq:    the prefill kernel's structure (128 query columns per workgroup, two 16-column
//          groups per wave, walk their key interval in 32-key steps through LDS), no running
//          maximum (lse is known); each column also computes its delta and lse * log2(e) and
//          writes lse * log2(e) and -delta to the workspace for the second launch (both
//          launches start the dout.v accumulators at -delta, so the MFMA yields dp - delta);
//   dk/dv: transposed roles: each workgroup holds 64 keys of one KV head in registers and
//          walks, for every query head of the group, the interval of targets whose supports
//          contain those keys (PBB: up to h(floor(s/h) + 2) - 1; SWA: s + W - 1).
// Every gradient element is written once, by the one workgroup that owns it (no atomics,
// deterministic).  Matrix-core products use v_mfma_f32_16x16x32_bf16 with the score layout of
// the forward (16 B-operand columns, 32 rows in two halves), P and dS rounded to bf16 as
// operands, fp32 accumulation, bf16 (RNE) outputs.

#include <type_traits>

#include "pbb_device.h"
#include "pbb_internal.h"

namespace pbb {
namespace {

// Waves per workgroup of the dq and dk/dv launches (16 kDqColGroups query columns or 16 keys
// per wave).
constexpr int kDqWaves = 4;
constexpr int kDqColGroups = 2;   // 16-column groups per dq wave
constexpr int kDkdvWaves = 4;
constexpr int kDkdvKeyGroups = 1;  // 16-key groups per dk/dv wave
constexpr int kDkdvWavesPerEU = 2; // occupancy the dk/dv register budget is set for

// Tiles read both as matrix-core row operands (16 bytes of one row per lane) and through
// transposed reads (4 rows x 8 bytes per 16 lanes) store 16-byte piece p of row r at p ^ g(r).
// g keeps both reads free of bank conflicts on gfx950's 64 LDS banks, where a 16-byte read
// serves, per cycle, the 16 lanes that share lane bit 5 and the parity of lane bits 2..4, and an
// 8-byte (or transposed) read the 32 lanes that share the parity of lane bits 3..5 (measured):
// within such a group, the row reads' pieces and the transposed reads' 8-byte units are all
// distinct with g(r) = 2 (r mod 8) for 256-byte rows and 2 ((r >> 1) mod 4) for 128-byte rows.
template <int D>
__device__ __forceinline__ int dual_swz(int r) {
  if constexpr (D == 128) return 2 * (r & 7);
  return 2 * ((r >> 1) & 3);
}

// Workgroup i runs on XCD i mod 8: give each XCD a contiguous run of tiles.
__device__ __forceinline__ int xcd_tile() {
  const int nblk = gridDim.x;
  const int per = nblk >> 3, rem = nblk & 7;
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  return (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + local;
}

// ------------------------------------------------------------------------------------------
// dq: 16 QC NW query columns (TQ positions x G heads, position-major) per workgroup; each wave
// owns QC groups of 16 columns, which share every K and V read of a step.
template <int D, int NW, int QC>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2)))
void bwd_dq_kernel(BackwardArgs a, int tq, int tiles) {
  constexpr int KK = D / 32, NB = D / 16, ROWB = D * 2, PPR = D / 8, RPI = 64 / PPR;
  constexpr int NG = 32 / RPI;           // 1 KiB DMA groups per 32-row tile
  constexpr int TILE = 32 * ROWB;
  constexpr int BUF = 2 * TILE;          // K tile, V tile (both in the dual layout)
  constexpr int STAGES = 3;
  constexpr int OPS = 2 * NG;
  constexpr int MYOPS = OPS / NW;
  static_assert(OPS % NW == 0 && MYOPS >= 1, "DMA split");
  __shared__ __align__(16) unsigned char smem[STAGES * BUF];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c16 = lane & 15, j4 = lane >> 4;
  const int G = a.group, n = a.n;
  const int tile_id = xcd_tile();
  const int bg = tile_id / tiles, tile = tile_id - bg * tiles;
  const int b = bg / a.hkv, g = bg - b * a.hkv;
  const int t0 = tile * tq;
  const int t_last = min(n - 1, t0 + tq - 1);
  const int kbeg = support_start(a.mode, a.block, a.window, t0);
  const int s_first = kbeg >> 5;
  const int nsteps = (t_last >> 5) - s_first + 1;
  const int mask_lo = support_start(a.mode, a.block, a.window, t_last);
  const int mask_hi = t0;

  const uint32_t rowstride = (uint32_t)a.hkv * ROWB;
  const unsigned char* kbase = (const unsigned char*)a.k + ((size_t)b * n * a.hkv + g) * ROWB;
  const unsigned char* vbase = (const unsigned char*)a.v + ((size_t)b * n * a.hkv + g) * ROWB;

  // This lane's query columns: column c -> position t0 + c / G, head g*G + c % G.
  int tc[QC], hc[QC], lo_c[QC], hi_c[QC];
  bool valid[QC];
  float lse2[QC], ndl[QC];  // lse * log2(e) and -delta of each column
  bf16x8 qB[QC][KK], gB[QC][KK], oB[QC][KK];
#pragma unroll
  for (int qc = 0; qc < QC; ++qc) {
    const int col = (wave * QC + qc) * 16 + c16;
    const int cp = col / G;
    tc[qc] = t0 + cp;
    hc[qc] = g * G + (col - cp * G);
    valid[qc] = cp < tq && tc[qc] < n;
    lo_c[qc] = valid[qc] ? support_start(a.mode, a.block, a.window, tc[qc]) : 0x7fffffff;
    hi_c[qc] = valid[qc] ? tc[qc] : -1;
    const size_t rowq = ((size_t)b * n + (valid[qc] ? tc[qc] : t0)) * a.hq + hc[qc];
    const uint16_t* qrow = (const uint16_t*)a.q + rowq * D;
    const uint16_t* grow = (const uint16_t*)a.dout + rowq * D;
    const uint16_t* orow = (const uint16_t*)a.out + rowq * D;
    const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const u32x4 wq = *(const u32x4*)(qrow + 32 * kk + 8 * j4);
      const u32x4 wg = *(const u32x4*)(grow + 32 * kk + 8 * j4);
      const u32x4 wo = *(const u32x4*)(orow + 32 * kk + 8 * j4);
      qB[qc][kk] = __builtin_bit_cast(bf16x8, valid[qc] ? wq : zero);
      gB[qc][kk] = __builtin_bit_cast(bf16x8, valid[qc] ? wg : zero);
      oB[qc][kk] = __builtin_bit_cast(bf16x8, valid[qc] ? wo : zero);
    }
    const float l = a.lse[((size_t)b * a.hq + hc[qc]) * n + (valid[qc] ? tc[qc] : t0)];
    lse2[qc] = valid[qc] ? l * 1.4426950408889634f : 0.0f;
  }

  // DMA of key step st: rows k0 .. k0+31 of K then V (wave-uniform base at row k0, lane offset
  // row * rowstride + piece); rows past t_last read the last piece of row t_last instead
  // (masked, and inside the tensor).
  uint32_t doff[MYOPS];
#pragma unroll
  for (int o = 0; o < MYOPS; ++o) {
    const int op = wave * MYOPS + o;
    const int x = op >= NG ? op - NG : op;
    const int row = x * RPI + lane / PPR;
    doff[o] = (uint32_t)row * rowstride + (uint32_t)(((lane % PPR) ^ dual_swz<D>(row)) * 16);
  }
  auto issue = [&](int stage, int st) {
    unsigned char* tp = smem + stage * BUF;
    const int k0 = (s_first + st) * 32;
    const uint32_t lim = (uint32_t)min(t_last - k0, 31) * rowstride + (ROWB - 16);
#pragma unroll
    for (int o = 0; o < MYOPS; ++o) {
      const int op = wave * MYOPS + o;
      const bool isv = op >= NG;
      const int x = isv ? op - NG : op;
      dma16((isv ? vbase : kbase) + (size_t)k0 * rowstride, min(doff[o], lim),
            tp + (isv ? TILE : 0) + x * 1024);
    }
  };

  // LDS offsets of this lane: row-operand reads (row c16, piece 4kk + j4; row 16 + c16 and
  // the V tile at fixed distances) and transposed reads of the K tile for chunk nb (row
  // 4j + c/4, channels 16nb + 4(c mod 4) .. +3).
  uint32_t roff[KK], kaddr[NB];
  {
    const uint32_t base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)smem;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
      roff[kk] = base + c16 * ROWB + (((4 * kk + j4) ^ dual_swz<D>(c16)) << 4);
    const int r = 4 * j4 + (c16 >> 2);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int p = 2 * nb + ((c16 & 3) >> 1);
      kaddr[nb] = base + r * ROWB + ((p ^ dual_swz<D>(r)) << 4) + ((c16 & 1) << 3);
    }
  }
  const __attribute__((address_space(3))) unsigned char* lds0 = nullptr;

  f32x4 acc[QC][NB];
#pragma unroll
  for (int qc = 0; qc < QC; ++qc)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[qc][nb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  const float c = a.scale_log2;

  issue(0, 0);
  if (nsteps > 1) issue(1, 1);
  int rstage = 0;

  // delta = dout . out of each column (the four quarters j hold channel slices 8j.. of every
  // 32-channel block), and lse * log2(e): -delta and lse * log2(e) are kept in registers for dq
  // and written to the workspace for the dk/dv launch.
#pragma unroll
  for (int qc = 0; qc < QC; ++qc) {
    float part = 0.0f;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
#pragma unroll
      for (int e = 0; e < 8; ++e)
        part = __builtin_fmaf((float)gB[qc][kk][e], (float)oB[qc][kk][e], part);
    ndl[qc] = -sum_xor16_32(part);
    if (valid[qc] && j4 == 0) {
      float* w = a.ws + ((size_t)b * a.hq + hc[qc]) * 2 * n + tc[qc];
      w[0] = lse2[qc];
      w[n] = ndl[qc];
    }
  }

  auto step = [&](int st, auto masked) {
    if (st + 1 < nsteps)
      __builtin_amdgcn_s_waitcnt(0x0F70 | (MYOPS & 15) | ((MYOPS >> 4) << 14));
    else
      __builtin_amdgcn_s_waitcnt(0x0F70);
    lds_barrier();
    if (st + 2 < nsteps) issue(rstage == 0 ? 2 : rstage - 1, st + 2);
    __builtin_amdgcn_sched_barrier(0);
    const uint32_t sb = (uint32_t)(rstage * BUF);
    const int k0 = (s_first + st) * 32;
    f32x4 s0[QC], s1[QC], d0[QC], d1[QC];
#pragma unroll
    for (int qc = 0; qc < QC; ++qc) {
      s0[qc] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      s1[qc] = s0[qc];
      d0[qc] = f32x4{ndl[qc], ndl[qc], ndl[qc], ndl[qc]};  // the products land on -delta
      d1[qc] = d0[qc];
    }
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const auto* p = lds0 + roff[kk] + sb;
      const bf16x8 ka = *(const __attribute__((address_space(3))) bf16x8*)(p);
      const bf16x8 kb = *(const __attribute__((address_space(3))) bf16x8*)(p + 16 * ROWB);
      const bf16x8 va = *(const __attribute__((address_space(3))) bf16x8*)(p + TILE);
      const bf16x8 vb = *(const __attribute__((address_space(3))) bf16x8*)(p + TILE + 16 * ROWB);
#pragma unroll
      for (int qc = 0; qc < QC; ++qc) {
        s0[qc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qB[qc][kk], s0[qc], 0, 0, 0);
        s1[qc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kb, qB[qc][kk], s1[qc], 0, 0, 0);
        d0[qc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, gB[qc][kk], d0[qc], 0, 0, 0);
        d1[qc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vb, gB[qc][kk], d1[qc], 0, 0, 0);
      }
    }
    // The K^T reads for dq go out now, under the softmax arithmetic.
    u32x2 kr[2 * NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      kr[2 * nb] = tr_read<0>(kaddr[nb] + sb);
      kr[2 * nb + 1] = tr_read<16 * ROWB>(kaddr[nb] + sb);
    }
    // ds = p (dp - delta) (the accumulators started at -delta), p = exp2(s c - lse2); masked
    // keys give p = 0.
    bf16x8 dsB[QC];
#pragma unroll
    for (int qc = 0; qc < QC; ++qc) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float sc = e < 4 ? s0[qc][e] : s1[qc][e - 4];
        const float dp = e < 4 ? d0[qc][e] : d1[qc][e - 4];
        float pe = fast_exp2(__builtin_fmaf(sc, c, -lse2[qc]));
        if constexpr (decltype(masked)::value) {
          const int key = k0 + (e < 4 ? 4 * j4 + e : 16 + 4 * j4 + (e - 4));
          pe = (key >= lo_c[qc] && key <= hi_c[qc]) ? pe : 0.0f;
        }
        dsB[qc][e] = (__bf16)(pe * dp);
      }
    }
    // dq^T += K^T ds^T.
    if constexpr (NB == 8) {
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(kr[0]), "+v"(kr[1]), "+v"(kr[2]), "+v"(kr[3]), "+v"(kr[4]),
                     "+v"(kr[5]), "+v"(kr[6]), "+v"(kr[7]), "+v"(kr[8]), "+v"(kr[9]),
                     "+v"(kr[10]), "+v"(kr[11]), "+v"(kr[12]), "+v"(kr[13]), "+v"(kr[14]),
                     "+v"(kr[15]));
    } else {
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(kr[0]), "+v"(kr[1]), "+v"(kr[2]), "+v"(kr[3]), "+v"(kr[4]),
                     "+v"(kr[5]), "+v"(kr[6]), "+v"(kr[7]));
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const u32x4 w = {kr[2 * nb][0], kr[2 * nb][1], kr[2 * nb + 1][0], kr[2 * nb + 1][1]};
#pragma unroll
      for (int qc = 0; qc < QC; ++qc)
        acc[qc][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, w),
                                                              dsB[qc], acc[qc][nb], 0, 0, 0);
    }
    rstage = rstage == STAGES - 1 ? 0 : rstage + 1;
    __builtin_amdgcn_sched_barrier(0);
  };

  int st_a = (mask_lo + 31) / 32 - s_first;
  int st_b = (mask_hi + 1) / 32 - s_first;
  st_a = max(0, min(st_a, nsteps));
  st_b = max(st_a, min(st_b, nsteps));
  for (int st = 0; st < st_a; ++st) step(st, std::true_type{});
  for (int st = st_a; st < st_b; ++st) step(st, std::false_type{});
  for (int st = st_b; st < nsteps; ++st) step(st, std::true_type{});

#pragma unroll
  for (int qc = 0; qc < QC; ++qc) {
    if (!valid[qc]) continue;
    uint16_t* drow = (uint16_t*)a.dq + (((size_t)b * n + tc[qc]) * a.hq + hc[qc]) * D;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      u32x2 w;
      w[0] = (uint32_t)float_to_bf16_rne(acc[qc][nb][0] * a.scale) |
             ((uint32_t)float_to_bf16_rne(acc[qc][nb][1] * a.scale) << 16);
      w[1] = (uint32_t)float_to_bf16_rne(acc[qc][nb][2] * a.scale) |
             ((uint32_t)float_to_bf16_rne(acc[qc][nb][3] * a.scale) << 16);
      *(u32x2*)(drow + 16 * nb + 4 * j4) = w;
    }
  }
}

// ------------------------------------------------------------------------------------------
// dk, dv: 16 KC NW keys of one KV head per workgroup (KC groups of 16 per wave, held as
// matrix-core B operands, sharing every Q and dout read of a step); the workgroup walks, for
// each query head of the group in turn, the 32-target steps of the targets whose supports
// contain its keys, through LDS: Q and dout rows (dual layout) and the steps' lse * log2(e)
// and -delta values.
template <int D, int NW, int KC, int WPE>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(WPE)))
void bwd_dkdv_kernel(BackwardArgs a, int tiles) {
  constexpr int KK = D / 32, NB = D / 16, ROWB = D * 2, PPR = D / 8, RPI = 64 / PPR;
  constexpr int NG = 32 / RPI;
  constexpr int TILE = 32 * ROWB;
  constexpr int BUF = 2 * TILE + 256;   // Q tile, dout tile, lse2[32] and -delta[32]
  constexpr int STAGES = 4;              // two stages of two target steps each
  constexpr int ROWOPS = 2 * NG;        // row DMAs per step; wave 0 also issues the lse/delta one
  constexpr int MYOPS = ROWOPS / NW;
  static_assert(ROWOPS % NW == 0 && MYOPS >= 1, "DMA split");
  constexpr int KT = 16 * KC * NW;      // keys per workgroup
  __shared__ __align__(16) unsigned char smem[STAGES * BUF];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c16 = lane & 15, j4 = lane >> 4;
  const int G = a.group, n = a.n;
  const int tile_id = xcd_tile();
  const int bg = tile_id / tiles, tile = tile_id - bg * tiles;
  const int b = bg / a.hkv, g = bg - b * a.hkv;
  const int s0k = tile * KT;                       // first key of the workgroup
  const int s1k = min(n - 1, s0k + KT - 1);        // last key
  const int q_first = s0k & ~31;                   // targets before s0k see none of these keys
  const int q_end = min(n - 1, support_last_target(a.mode, a.block, a.window, s1k));
  const int qsteps = (q_end >> 5) - (q_first >> 5) + 1;
  const int nsteps = G * qsteps;                    // (head, target step) pairs
  // Target steps j in [ja, jb) are interior for every head: all their targets come at or after
  // the last key and at or before the last target of the first key (the supports are
  // intervals ending at the target, so every pair is covered); a partial key tile has none.
  int ja = (s1k - q_first + 31) >> 5;
  const int lim_t = min(n - 1, support_last_target(a.mode, a.block, a.window, s0k)) - 31 - q_first;
  int jb = (lim_t < 0 || s1k - s0k + 1 != KT) ? 0 : (lim_t >> 5) + 1;
  ja = min(ja, qsteps);
  jb = max(ja, min(jb, qsteps));

  // This wave's keys as B operands: lane (key c16 of group kc, slice j) holds channels
  // 32kk + 8j .. +7.  Targets that see a key: key .. min(q_end, last target of the key).
  int key[KC], t_lo[KC], t_hi[KC];
  bool kvalid[KC];
  bf16x8 kB[KC][KK], vB[KC][KK];
#pragma unroll
  for (int kc = 0; kc < KC; ++kc) {
    key[kc] = s0k + (wave * KC + kc) * 16 + c16;
    kvalid[kc] = key[kc] < n;
    t_lo[kc] = kvalid[kc] ? key[kc] : 0x7fffffff;
    t_hi[kc] = min(q_end, support_last_target(a.mode, a.block, a.window, key[kc]));
    const size_t rowk = ((size_t)b * n + (kvalid[kc] ? key[kc] : s0k)) * a.hkv + g;
    const uint16_t* krow = (const uint16_t*)a.k + rowk * D;
    const uint16_t* vrow = (const uint16_t*)a.v + rowk * D;
    const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const u32x4 wk = *(const u32x4*)(krow + 32 * kk + 8 * j4);
      const u32x4 wv = *(const u32x4*)(vrow + 32 * kk + 8 * j4);
      kB[kc][kk] = __builtin_bit_cast(bf16x8, kvalid[kc] ? wk : zero);
      vB[kc][kk] = __builtin_bit_cast(bf16x8, kvalid[kc] ? wv : zero);
    }
  }

  // DMA of (head hi, target step j): rows q0 .. q0+31 of Q and dout (wave-uniform base, lane
  // offset row * qrowstride + piece; rows past q_end read the last piece of row q_end), and,
  // from wave 0, lse2 (lanes 0..31) and -delta (lanes 32..63) of the same targets.
  const uint32_t qrowstride = (uint32_t)a.hq * ROWB;
  const unsigned char* qb0 = (const unsigned char*)a.q + ((size_t)b * n * a.hq + g * G) * ROWB;
  const unsigned char* gb0 = (const unsigned char*)a.dout + ((size_t)b * n * a.hq + g * G) * ROWB;
  const float* wb0 = a.ws + ((size_t)b * a.hq + g * G) * 2 * n;
  uint32_t doff[MYOPS];
#pragma unroll
  for (int o = 0; o < MYOPS; ++o) {
    const int op = wave * MYOPS + o;
    const int x = op >= NG ? op - NG : op;
    const int row = x * RPI + lane / PPR;
    doff[o] = (uint32_t)row * qrowstride + (uint32_t)(((lane % PPR) ^ dual_swz<D>(row)) * 16);
  }
  auto issue = [&](int stage, int hi, int j) {
    unsigned char* tp = smem + stage * BUF;
    const int q0 = q_first + 32 * j;
    const int last = min(q_end - q0, 31);
    const uint32_t lim = (uint32_t)last * qrowstride + (ROWB - 16);
    const size_t rowbase = ((size_t)q0 * a.hq + hi) * ROWB;
#pragma unroll
    for (int o = 0; o < MYOPS; ++o) {
      const int op = wave * MYOPS + o;
      const bool isg = op >= NG;
      const int x = isg ? op - NG : op;
      dma16((isg ? gb0 : qb0) + rowbase, min(doff[o], lim), tp + (isg ? TILE : 0) + x * 1024);
    }
    if (wave == 0) {
      const float* s = wb0 + (size_t)hi * 2 * n + q0 + min(lane & 31, last) + (lane >> 5) * n;
      __builtin_amdgcn_global_load_lds((const void*)s,
                                       (__attribute__((address_space(3))) void*)(tp + 2 * TILE),
                                       4, 0, 0);
    }
  };

  // LDS offsets of this lane: row-operand reads of the Q tile (row c16, piece 4kk + j4; row
  // 16 + c16 and the dout tile at fixed distances) and transposed reads for chunk nb.
  uint32_t roff[KK], taddr[NB];
  {
    const uint32_t base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)smem;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
      roff[kk] = base + c16 * ROWB + (((4 * kk + j4) ^ dual_swz<D>(c16)) << 4);
    const int r = 4 * j4 + (c16 >> 2);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int p = 2 * nb + ((c16 & 3) >> 1);
      taddr[nb] = base + r * ROWB + ((p ^ dual_swz<D>(r)) << 4) + ((c16 & 1) << 3);
    }
  }
  const uint32_t lbase =
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)smem + 2 * TILE;
  const __attribute__((address_space(3))) unsigned char* lds0 = nullptr;

  f32x4 acck[KC][NB], accv[KC][NB];
#pragma unroll
  for (int kc = 0; kc < KC; ++kc)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      acck[kc][nb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      accv[kc][nb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    }
  const float c = a.scale_log2;

  // Issue cursor (head, step): the next target step to load.
  int ih = 0, ij = 0;
  auto advance = [&]() {
    if (++ij == qsteps) {
      ij = 0;
      ++ih;
    }
  };
  issue(0, ih, ij);
  advance();
  if (nsteps > 1) {
    issue(1, ih, ij);
    advance();
  }

  auto step = [&](int gs, int j, auto masked) {
    // Target steps go in pairs (buffers 0-1 and 2-3): at the start of a pair this wave's loads
    // of both steps have landed; one barrier makes every wave's share visible and frees the
    // other pair's buffers (every wave has finished the previous pair), and the next pair is
    // issued into them -- one barrier per two steps (measured 2-4 % faster than one per step).
    if ((gs & 1) == 0) {
      __builtin_amdgcn_s_waitcnt(0x0F70);
      lds_barrier();
      const int ob = ((gs >> 1) & 1) ? 0 : 2;
      if (gs + 2 < nsteps) {
        issue(ob, ih, ij);
        advance();
      }
      if (gs + 3 < nsteps) {
        issue(ob + 1, ih, ij);
        advance();
      }
    }
    const int rstage = ((gs >> 1) & 1) * 2 + (gs & 1);
    __builtin_amdgcn_sched_barrier(0);
    const uint32_t sb = (uint32_t)(rstage * BUF);
    const int q0 = q_first + 32 * j;
    // lse2 and -delta of this lane's 8 targets (rows 4j..4j+3 and 16+4j..16+4j+3).
    const auto* lp = lds0 + lbase + sb + 16 * j4;
    const f32x4 la = *(const __attribute__((address_space(3))) f32x4*)(lp);
    const f32x4 lb = *(const __attribute__((address_space(3))) f32x4*)(lp + 64);
    const f32x4 da = *(const __attribute__((address_space(3))) f32x4*)(lp + 128);
    const f32x4 db = *(const __attribute__((address_space(3))) f32x4*)(lp + 192);
    // Scores with targets on the rows (two halves of 16) and this wave's keys on the columns;
    // the dout.v products land on -delta of their target row.
    f32x4 s0[KC], s1[KC], d0[KC], d1[KC];
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
      s0[kc] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      s1[kc] = s0[kc];
      d0[kc] = da;
      d1[kc] = db;
    }
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const auto* p = lds0 + roff[kk] + sb;
      const bf16x8 qa = *(const __attribute__((address_space(3))) bf16x8*)(p);
      const bf16x8 qb = *(const __attribute__((address_space(3))) bf16x8*)(p + 16 * ROWB);
      const bf16x8 ga = *(const __attribute__((address_space(3))) bf16x8*)(p + TILE);
      const bf16x8 gb = *(const __attribute__((address_space(3))) bf16x8*)(p + TILE + 16 * ROWB);
#pragma unroll
      for (int kc = 0; kc < KC; ++kc) {
        s0[kc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa, kB[kc][kk], s0[kc], 0, 0, 0);
        s1[kc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qb, kB[kc][kk], s1[kc], 0, 0, 0);
        d0[kc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ga, vB[kc][kk], d0[kc], 0, 0, 0);
        d1[kc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(gb, vB[kc][kk], d1[kc], 0, 0, 0);
      }
    }
    // The dout^T reads for dv go out now, under the softmax arithmetic.
    u32x2 gr[2 * NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      gr[2 * nb] = tr_read<TILE>(taddr[nb] + sb);
      gr[2 * nb + 1] = tr_read<TILE + 16 * ROWB>(taddr[nb] + sb);
    }
    bf16x8 pB[KC], dsB[KC];
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float sc = e < 4 ? s0[kc][e] : s1[kc][e - 4];
        const float dp = e < 4 ? d0[kc][e] : d1[kc][e - 4];
        const float l2 = e < 4 ? la[e] : lb[e - 4];
        float pe = fast_exp2(__builtin_fmaf(sc, c, -l2));
        if constexpr (decltype(masked)::value) {
          const int t = q0 + (e < 4 ? 4 * j4 + e : 16 + 4 * j4 + (e - 4));
          pe = (t >= t_lo[kc] && t <= t_hi[kc]) ? pe : 0.0f;
        }
        pB[kc][e] = (__bf16)pe;
        dsB[kc][e] = (__bf16)(pe * dp);
      }
    }
    // dv^T += dout^T p, dk^T += Q^T ds: dout^T and Q^T by transposed reads.
    if constexpr (NB == 8) {
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(gr[0]), "+v"(gr[1]), "+v"(gr[2]), "+v"(gr[3]), "+v"(gr[4]),
                     "+v"(gr[5]), "+v"(gr[6]), "+v"(gr[7]), "+v"(gr[8]), "+v"(gr[9]),
                     "+v"(gr[10]), "+v"(gr[11]), "+v"(gr[12]), "+v"(gr[13]), "+v"(gr[14]),
                     "+v"(gr[15]));
    } else {
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(gr[0]), "+v"(gr[1]), "+v"(gr[2]), "+v"(gr[3]), "+v"(gr[4]),
                     "+v"(gr[5]), "+v"(gr[6]), "+v"(gr[7]));
    }
    // The Q^T reads go out before the dv products so that they overlap them.
    u32x2 qr[2 * NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      qr[2 * nb] = tr_read<0>(taddr[nb] + sb);
      qr[2 * nb + 1] = tr_read<16 * ROWB>(taddr[nb] + sb);
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const u32x4 w = {gr[2 * nb][0], gr[2 * nb][1], gr[2 * nb + 1][0], gr[2 * nb + 1][1]};
#pragma unroll
      for (int kc = 0; kc < KC; ++kc)
        accv[kc][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, w),
                                                               pB[kc], accv[kc][nb], 0, 0, 0);
    }
    if constexpr (NB == 8) {
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(qr[0]), "+v"(qr[1]), "+v"(qr[2]), "+v"(qr[3]), "+v"(qr[4]),
                     "+v"(qr[5]), "+v"(qr[6]), "+v"(qr[7]), "+v"(qr[8]), "+v"(qr[9]),
                     "+v"(qr[10]), "+v"(qr[11]), "+v"(qr[12]), "+v"(qr[13]), "+v"(qr[14]),
                     "+v"(qr[15]));
    } else {
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(qr[0]), "+v"(qr[1]), "+v"(qr[2]), "+v"(qr[3]), "+v"(qr[4]),
                     "+v"(qr[5]), "+v"(qr[6]), "+v"(qr[7]));
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const u32x4 w = {qr[2 * nb][0], qr[2 * nb][1], qr[2 * nb + 1][0], qr[2 * nb + 1][1]};
#pragma unroll
      for (int kc = 0; kc < KC; ++kc)
        acck[kc][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, w),
                                                               dsB[kc], acck[kc][nb], 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  };

  int gs = 0;
  for (int hi = 0; hi < G; ++hi) {
    for (int j = 0; j < ja; ++j, ++gs) step(gs, j, std::true_type{});
    for (int j = ja; j < jb; ++j, ++gs) step(gs, j, std::false_type{});
    for (int j = jb; j < qsteps; ++j, ++gs) step(gs, j, std::true_type{});
  }

#pragma unroll
  for (int kc = 0; kc < KC; ++kc) {
    if (!kvalid[kc]) continue;
    const size_t rowk = ((size_t)b * n + key[kc]) * a.hkv + g;
    uint16_t* dkrow = (uint16_t*)a.dk + rowk * D;
    uint16_t* dvrow = (uint16_t*)a.dv + rowk * D;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      u32x2 wk, wv;
      wk[0] = (uint32_t)float_to_bf16_rne(acck[kc][nb][0] * a.scale) |
              ((uint32_t)float_to_bf16_rne(acck[kc][nb][1] * a.scale) << 16);
      wk[1] = (uint32_t)float_to_bf16_rne(acck[kc][nb][2] * a.scale) |
              ((uint32_t)float_to_bf16_rne(acck[kc][nb][3] * a.scale) << 16);
      wv[0] = (uint32_t)float_to_bf16_rne(accv[kc][nb][0]) |
              ((uint32_t)float_to_bf16_rne(accv[kc][nb][1]) << 16);
      wv[1] = (uint32_t)float_to_bf16_rne(accv[kc][nb][2]) |
              ((uint32_t)float_to_bf16_rne(accv[kc][nb][3]) << 16);
      *(u32x2*)(dkrow + 16 * nb + 4 * j4) = wk;
      *(u32x2*)(dvrow + 16 * nb + 4 * j4) = wv;
    }
  }
}

template <int D>
hipError_t launch_backward_d(const BackwardArgs& a, hipStream_t stream) {
  const int tq = (16 * kDqColGroups * kDqWaves) / a.group;
  const int qtiles = (a.n + tq - 1) / tq;
  hipLaunchKernelGGL((bwd_dq_kernel<D, kDqWaves, kDqColGroups>),
                     dim3((unsigned)((size_t)a.batch * a.hkv * qtiles)), dim3(kDqWaves * 64), 0,
                     stream, a, tq, qtiles);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  constexpr int KT = 16 * kDkdvKeyGroups * kDkdvWaves;
  const int ktiles = (a.n + KT - 1) / KT;
  hipLaunchKernelGGL((bwd_dkdv_kernel<D, kDkdvWaves, kDkdvKeyGroups, kDkdvWavesPerEU>),
                     dim3((unsigned)((size_t)a.batch * a.hkv * ktiles)), dim3(kDkdvWaves * 64), 0,
                     stream, a, ktiles);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_backward_bf16(const BackwardArgs& a, int32_t head_dim, hipStream_t stream) {
  return head_dim == 128 ? launch_backward_d<128>(a, stream) : launch_backward_d<64>(a, stream);
}

}  // namespace pbb
