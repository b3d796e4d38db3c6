// HIP prefill kernel for Post-Boundary Bridge (PBB) attention on gfx950 (MI355X, CDNA4).
//
// Every position t = 0..n-1 of a prompt attends with one softmax over its own support
// (Sec. 3, Eq.(pbb) and Eq.(attention)).  With h = B/2 that support is the interval
// [a(t), t], a(t) = max(0, h*(floor(t/h) - 1)) (Sec. 3 "Flash-PBB"; Appendix A.3): the causal
// block prefix plus, for the first h phases of a block, the preceding half-block, i.e. causal
// block tiles plus h x h bridge rectangles (Appendix F.4), never a dense n x n mask.  The
// sliding-window variant uses [max(0, t-W+1), t] (Prop. 2).  a(t) never decreases, so the
// keys any run of consecutive positions needs form one interval.
//
// Work unit: TQ = floor(16*QC*NW / G) consecutive positions of one (sequence, KV head) with
// all G query heads of that KV head, i.e. 16*QC*NW query columns ordered position-major,
// head-minor (native grouped-query attention: the K/V tile is read once for the group).
// Keys of the unit's interval stream through LDS in 32-key steps, three stages deep, each
// tile loaded once per workgroup by LDS DMA and shared by the 4 waves; each wave owns QC
// groups of 16 columns.  Per step a wave computes S^T = K Q^T and O^T += V^T P^T on
// v_mfma_f32_16x16x32_bf16 exactly as the decode kernel does, the 16 B-operand columns being
// 16 queries; per-column bounds mask the tile; the online softmax keeps fp32 running
// maxima and sums (the log-sum-exp rescaling of Appendix A.4, Eq.(lse)).  Outputs are rounded
// to bf16 (RNE); the log-partition is written in natural-log units.  Finally every workgroup
// copies those of its positions that fall in the last `slots` positions of the prompt into the
// ring (slot s mod slots, Appendix F.1), the state decode continues from.

#include <type_traits>

#include "pbb_device.h"
#include "pbb_internal.h"

namespace pbb {
namespace {

// Waves per workgroup, 16-column groups per wave and LDS stages (d = 128, d = 64).
constexpr int kPrefillWaves128 = 4;
constexpr int kPrefillWaves64 = 4;
constexpr int kPrefillStages128 = 3;
constexpr int kPrefillStages64 = 5;  // a tile at d = 64 walks few key steps: all in flight early
constexpr int kPrefillColGroups128 = 2;
constexpr int kPrefillColGroups64 = 2;

// Starting reference of the running maximum (log2 units): finite and below any score.
constexpr float kNoScore = -1.0e30f;

__device__ __forceinline__ int support_lo(const PrefillArgs& a, int t) {
  return support_start(a.mode, a.block, a.window, t);
}

// Three waves per SIMD (three workgroups of 48 KiB LDS per CU): the register budget this sets
// at d = 128 (168) leaves a few values of the epilogue in scratch, outside the key loop.
template <int D, int QC, int NW, int ST>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(3)))
void prefill_bf16_kernel(PrefillArgs a, int tq, int tiles) {
  constexpr int KK = D / 32;            // 32-channel slices of the score contraction
  constexpr int NB = D / 16;            // 16-channel blocks of the output
  constexpr int ROWB = D * 2;           // bytes of one K or V row
  constexpr int PPR = D / 8;            // 16-byte pieces per row
  constexpr int RPI = 64 / PPR;         // rows per 1 KiB DMA group
  constexpr int NG = 32 / RPI;          // DMA groups per step and tensor
  constexpr int KTILE = 32 * ROWB;
  constexpr int VTILE = 32 * ROWB;
  constexpr int BUF = KTILE + VTILE;
  constexpr int STAGES = ST;
  static_assert(STAGES >= 3 && STAGES <= 5, "stages");
  constexpr int OPS = 2 * NG;           // DMA instructions per step (K tile, then V tile)
  constexpr int MYOPS = OPS / NW;       // issued by each wave
  static_assert(OPS % NW == 0, "DMA split");
  __shared__ __align__(256) unsigned char smem[STAGES * BUF];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c16 = lane & 15;
  const int j4 = lane >> 4;
  const int G = a.group;
  const int n = a.n;

  // Workgroup i runs on XCD i mod 8; give each XCD a contiguous run of tiles so that tiles
  // sharing keys (neighbours of one sequence and KV head) share that XCD's L2.
  const int nblk = gridDim.x;
  const int per = nblk >> 3, rem = nblk & 7;
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int tile_id = (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + local;
  const int bg = tile_id / tiles;
  const int tile = tile_id - bg * tiles;
  const int b = bg / a.hkv;
  const int g = bg - b * a.hkv;
  const int t0 = tile * tq;
  const int t_last = min(n - 1, t0 + tq - 1);
  const int kbeg = support_lo(a, t0);
  const int s_first = kbeg >> 5;
  const int nsteps = (t_last >> 5) - s_first + 1;
  // Keys [mask_lo, mask_hi] are in the support of every position of the tile (a(t) never
  // decreases): steps inside that range need no masking.
  const int mask_lo = support_lo(a, t_last);
  const int mask_hi = t0;

  const uint32_t rowstride = (uint32_t)a.hkv * ROWB;  // bytes between consecutive positions
  const unsigned char* kbase = (const unsigned char*)a.k + ((size_t)b * n * a.hkv + g) * ROWB;
  const unsigned char* vbase = (const unsigned char*)a.v + ((size_t)b * n * a.hkv + g) * ROWB;

  // This lane's query columns: column c -> position t0 + c / G, head g*G + c % G.
  int lo_c[QC], hi_c[QC], tcol[QC], hcol[QC];
  bool valid[QC];
  bf16x8 qB[QC][KK];
#pragma unroll
  for (int qc = 0; qc < QC; ++qc) {
    const int col = (wave * QC + qc) * 16 + c16;
    const int cp = col / G;
    tcol[qc] = t0 + cp;
    hcol[qc] = g * G + (col - cp * G);
    valid[qc] = cp < tq && tcol[qc] < n;
    lo_c[qc] = valid[qc] ? support_lo(a, tcol[qc]) : 0x7fffffff;
    hi_c[qc] = valid[qc] ? tcol[qc] : -1;
    const uint16_t* qrow = (const uint16_t*)a.q +
        ((size_t)(b * (size_t)n + (valid[qc] ? tcol[qc] : t0)) * a.hq + hcol[qc]) * D;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const u32x4 w = *(const u32x4*)(qrow + 32 * kk + 8 * j4);
      const u32x4 zero = {0u, 0u, 0u, 0u};
      qB[qc][kk] = __builtin_bit_cast(bf16x8, valid[qc] ? w : zero);
    }
  }

  auto swz_k = [](int r) -> int { return D == 128 ? (r & 15) : ((r >> 1) & 7); };
  // V rows: 16-byte piece p of row r at p ^ swz_v(r).  The transposed reads below (4 rows x
  // 8 bytes per 16 lanes) then hit distinct banks within every group of 32 lanes that an 8-byte
  // LDS read serves per cycle on gfx950 (the lanes sharing the parity of lane bits 3..5).
  auto swz_v = [](int r) -> int { return D == 128 ? 2 * (r & 7) : 2 * ((r >> 1) & 3); };
  // LDS byte addresses of this lane's reads in stage 0: K rows c16 (and 16 + c16, a fixed
  // distance on) at piece 4kk + j4, and the transposed V reads of chunk nb: row 4j4 + c16/4,
  // channels 16nb + 4(c16 mod 4) .. +3 (rows 16.. a fixed distance on).  For d = 128, chunk
  // nb + 4 sits at the byte offset of chunk nb with bit 7 flipped (rows are 256-byte aligned).
  uint32_t kaddr[KK], vaddr[4];
  {
    const uint32_t base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)smem;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
      kaddr[kk] = base + c16 * ROWB + (((4 * kk + j4) ^ swz_k(c16)) << 4);
    const int vrow = 4 * j4 + (c16 >> 2);
#pragma unroll
    for (int q = 0; q < 4; ++q)
      vaddr[q] = base + KTILE + vrow * ROWB +
                 (((2 * q + ((c16 & 3) >> 1)) ^ swz_v(vrow)) << 4) + ((c16 & 1) << 3);
  }
  const __attribute__((address_space(3))) unsigned char* lds0 = nullptr;

  // This wave's share of the DMA of a step: MYOPS 1 KiB pieces, each lane one 16-byte piece of
  // one key row, addressed as a wave-uniform base (the step's first key row) plus a 32-bit lane
  // offset.  In the last step, rows past t_last read the last piece of row t_last instead
  // (inside the tensor; masked for every column).
  uint32_t doff[MYOPS];
#pragma unroll
  for (int o = 0; o < MYOPS; ++o) {
    const int op = wave * MYOPS + o;
    const bool isv = op >= NG;
    const int x = isv ? op - NG : op;
    const int row = x * RPI + lane / PPR;
    const int piece = (lane % PPR) ^ (isv ? swz_v(row) : swz_k(row));
    doff[o] = (uint32_t)row * rowstride + (uint32_t)(piece * 16);
  }
  auto issue = [&](int stage, int st) {
    unsigned char* tile_p = smem + stage * BUF;
    const int k0 = (s_first + st) * 32;
    const uint32_t lim = (uint32_t)min(t_last - k0, 31) * rowstride + (ROWB - 16);
#pragma unroll
    for (int o = 0; o < MYOPS; ++o) {
      const int op = wave * MYOPS + o;
      const bool isv = op >= NG;
      const int x = isv ? op - NG : op;
      dma16((isv ? vbase : kbase) + (size_t)k0 * rowstride, min(doff[o], lim),
            tile_p + (isv ? KTILE : 0) + x * 1024);
    }
  };

  // m starts at a finite floor below any score, so that a column whose keys are all masked so
  // far gets exp2(-inf - m) = 0 without a separate test; its first real maximum always moves m.
  float m[QC], lsum[QC];
  f32x4 acc[QC][NB];
#pragma unroll
  for (int qc = 0; qc < QC; ++qc) {
    m[qc] = kNoScore;
    lsum[qc] = 0.0f;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[qc][nb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  }

  // Steps 0 .. STAGES-2 go out first; step st then issues step st + STAGES - 1.
#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (s < nsteps) issue(s, s);
  int rstage = 0;
  constexpr int W1 = 0x0F70 | (MYOPS & 15) | ((MYOPS >> 4) << 14);
  constexpr int W2 = 0x0F70 | ((2 * MYOPS) & 15) | (((2 * MYOPS) >> 4) << 14);
  constexpr int W3 = 0x0F70 | ((3 * MYOPS) & 15) | (((3 * MYOPS) >> 4) << 14);

  auto step = [&](int st, auto masked) {
    // This wave's loads of step st have landed once at most the loads of the steps issued
    // after it (up to STAGES - 2) are outstanding; the barrier then covers every wave's loads,
    // and every wave is done with step st-1, whose stage the loads of step st+STAGES-1 reuse.
    const int ahead = min(STAGES - 2, nsteps - 1 - st);
    if (ahead >= 3) __builtin_amdgcn_s_waitcnt(W3);
    else if (ahead == 2) __builtin_amdgcn_s_waitcnt(W2);
    else if (ahead == 1) __builtin_amdgcn_s_waitcnt(W1);
    else __builtin_amdgcn_s_waitcnt(0x0F70);
    lds_barrier();
    if (st + STAGES - 1 < nsteps)
      issue(rstage == 0 ? STAGES - 1 : rstage - 1, st + STAGES - 1);
    __builtin_amdgcn_sched_barrier(0);

    const uint32_t sb = (uint32_t)(rstage * BUF);
    const int k0 = (s_first + st) * 32;
    f32x4 s0[QC], s1[QC];
#pragma unroll
    for (int qc = 0; qc < QC; ++qc) {
      s0[qc] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      s1[qc] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    }
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const auto* kp = lds0 + kaddr[kk] + sb;
      const bf16x8 ka = *(const __attribute__((address_space(3))) bf16x8*)(kp);
      const bf16x8 kb = *(const __attribute__((address_space(3))) bf16x8*)(kp + 16 * ROWB);
#pragma unroll
      for (int qc = 0; qc < QC; ++qc) {
        s0[qc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qB[qc][kk], s0[qc], 0, 0, 0);
        s1[qc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kb, qB[qc][kk], s1[qc], 0, 0, 0);
      }
    }
    // Online softmax in log2 units with a lazily moved reference m (the log-sum-exp rescaling
    // of Eq.(lse)): the weights are taken against the current m, and m moves to the column
    // maxima (the accumulators rescaled, the weights taken again) only in a step where the
    // eight weights of some lane and column sum above 2^8 or to infinity: a column's first
    // step with a real score (m starts at a finite floor), any step in which a score rises
    // more than 8 log2 units above m, and steps where several rise more than 5.  No other step
    // computes a maximum.  The result is the same softmax (numerator and denominator share
    // every reference change), and the weights that enter the sums and products stay <= 2^8.
    const float c = a.scale_log2;
    bf16x8 pB[QC];
    float ps[QC];
    if constexpr (decltype(masked)::value) {
#pragma unroll
      for (int qc = 0; qc < QC; ++qc)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int key = k0 + (e < 4 ? 4 * j4 + e : 16 + 4 * j4 + (e - 4));
          const bool in = key >= lo_c[qc] && key <= hi_c[qc];
          if (e < 4) s0[qc][e] = in ? s0[qc][e] : kNegInf;
          else s1[qc][e - 4] = in ? s1[qc][e - 4] : kNegInf;
        }
    }
    auto weights = [&]() {
      bool over = false;
#pragma unroll
      for (int qc = 0; qc < QC; ++qc) {
        float sum = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float sc = e < 4 ? s0[qc][e] : s1[qc][e - 4];
          const float pe = fast_exp2(__builtin_fmaf(sc, c, -m[qc]));
          sum += pe;
          pB[qc][e] = (__bf16)pe;
        }
        ps[qc] = sum;
        over |= !(sum <= kWeightCap);
      }
      return over;
    };
    auto move_reference = [&]() {
#pragma unroll
      for (int qc = 0; qc < QC; ++qc) {
        float mx = kNegInf;
#pragma unroll
        for (int e = 0; e < 8; ++e) mx = fmaxf(mx, e < 4 ? s0[qc][e] : s1[qc][e - 4]);
        const float cand = max_xor16_32(mx) * c;
        const bool grow = cand > m[qc];
        const float alpha = grow ? fast_exp2(m[qc] - cand) : 1.0f;
        m[qc] = grow ? cand : m[qc];
        lsum[qc] *= alpha;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[qc][nb] *= alpha;
      }
    };
    // The first step sets the reference before its weights (it would always move it).
    if (st == 0) move_reference();
    if (__builtin_amdgcn_ballot_w64(weights()) != 0) {
      move_reference();
      weights();
    }
#pragma unroll
    for (int qc = 0; qc < QC; ++qc) lsum[qc] += ps[qc];
    // V^T operand of O^T += V^T P^T: lane (c16, j4) needs channel 16nb + c16 of keys
    // 4j4..4j4+3 and 16+4j4..16+4j4+3 (the key order of P^T in the score layout).  One
    // transposed read per half: within each 16-lane group, lane i names 4 channels
    // 16nb + 4(i mod 4) .. +3 of key row 4j4 + i/4, and lane c16 receives channel 16nb + c16 of
    // those four rows.
    u32x2 vr[2 * NB];
    constexpr int HI = 16 * ROWB;   // rows 16.. of the tile
    vr[0] = tr_read<0>(vaddr[0] + sb);
    vr[1] = tr_read<HI>(vaddr[0] + sb);
    vr[2] = tr_read<0>(vaddr[1] + sb);
    vr[3] = tr_read<HI>(vaddr[1] + sb);
    vr[4] = tr_read<0>(vaddr[2] + sb);
    vr[5] = tr_read<HI>(vaddr[2] + sb);
    vr[6] = tr_read<0>(vaddr[3] + sb);
    vr[7] = tr_read<HI>(vaddr[3] + sb);
    if constexpr (NB == 8) {
      vr[8] = tr_read<0>((vaddr[0] ^ 128u) + sb);
      vr[9] = tr_read<HI>((vaddr[0] ^ 128u) + sb);
      vr[10] = tr_read<0>((vaddr[1] ^ 128u) + sb);
      vr[11] = tr_read<HI>((vaddr[1] ^ 128u) + sb);
      vr[12] = tr_read<0>((vaddr[2] ^ 128u) + sb);
      vr[13] = tr_read<HI>((vaddr[2] ^ 128u) + sb);
      vr[14] = tr_read<0>((vaddr[3] ^ 128u) + sb);
      vr[15] = tr_read<HI>((vaddr[3] ^ 128u) + sb);
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
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const u32x4 w = {vr[2 * nb][0], vr[2 * nb][1], vr[2 * nb + 1][0], vr[2 * nb + 1][1]};
      const bf16x8 va = __builtin_bit_cast(bf16x8, w);
#pragma unroll
      for (int qc = 0; qc < QC; ++qc)
        acc[qc][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pB[qc], acc[qc][nb], 0, 0, 0);
    }
    rstage = rstage == STAGES - 1 ? 0 : rstage + 1;
    __builtin_amdgcn_sched_barrier(0);
  };

  // Steps whose 32 keys all lie in every position's support need no mask: they form one run
  // [st_a, st_b); the steps before (a ragged interval start) and after (the causal diagonal)
  // are masked.
  int st_a = (mask_lo + 31) / 32 - s_first;
  int st_b = (mask_hi + 1) / 32 - s_first;
  st_a = max(0, min(st_a, nsteps));
  st_b = max(st_a, min(st_b, nsteps));
  for (int st = 0; st < st_a; ++st) step(st, std::true_type{});
  for (int st = st_a; st < st_b; ++st) step(st, std::false_type{});
  for (int st = st_b; st < nsteps; ++st) step(st, std::true_type{});

  // Outputs: o = acc / l (bf16 RNE), lse = (m + log2 l) * ln 2.
#pragma unroll
  for (int qc = 0; qc < QC; ++qc) {
    const float l = sum_xor16_32(lsum[qc]);
    if (!valid[qc]) continue;
    const float inv = 1.0f / l;
    uint16_t* orow = (uint16_t*)a.out + ((size_t)(b * (size_t)n + tcol[qc]) * a.hq + hcol[qc]) * D;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      u32x2 w;
      w[0] = (uint32_t)float_to_bf16_rne(acc[qc][nb][0] * inv) |
             ((uint32_t)float_to_bf16_rne(acc[qc][nb][1] * inv) << 16);
      w[1] = (uint32_t)float_to_bf16_rne(acc[qc][nb][2] * inv) |
             ((uint32_t)float_to_bf16_rne(acc[qc][nb][3] * inv) << 16);
      *(u32x2*)(orow + 16 * nb + 4 * j4) = w;
    }
    if (a.lse != nullptr && j4 == 0)
      a.lse[((size_t)b * a.hq + hcol[qc]) * n + tcol[qc]] =
          (m[qc] + __builtin_log2f(l)) * 0.69314718055994531f;
  }

  // Ring state after the prompt: positions max(0, n - slots) .. n-1 at slot s mod slots.
  if (a.k_ring != nullptr) {
    const int first = max(t0, n - a.slots);
    const int count = t_last - first + 1;
    for (int idx = tid; idx < 2 * count * PPR; idx += NW * 64) {
      const int which = idx / (count * PPR);
      const int rest = idx - which * count * PPR;
      const int t = first + rest / PPR;
      const int pc = rest % PPR;
      const unsigned char* src = (which ? vbase : kbase) + (size_t)t * rowstride + pc * 16;
      unsigned char* dst = (unsigned char*)(which ? a.v_ring : a.k_ring) +
                           ((size_t)bg * a.slots + (t % a.slots)) * ROWB + pc * 16;
      *(u32x4*)dst = *(const u32x4*)src;
    }
  }
}

template <int D>
hipError_t launch_prefill_d(const PrefillArgs& a, hipStream_t stream) {
  constexpr int QC = D == 128 ? kPrefillColGroups128 : kPrefillColGroups64;
  constexpr int NW = D == 128 ? kPrefillWaves128 : kPrefillWaves64;
  constexpr int ST = D == 128 ? kPrefillStages128 : kPrefillStages64;
  const int tq = 16 * QC * NW / a.group;
  const int tiles = (a.n + tq - 1) / tq;
  const size_t blocks = (size_t)a.batch * a.hkv * tiles;
  if (blocks == 0) return hipSuccess;
  if (blocks > 0x7fffffffull) return hipErrorInvalidValue;
  hipLaunchKernelGGL((prefill_bf16_kernel<D, QC, NW, ST>), dim3((unsigned)blocks),
                     dim3(NW * 64), 0, stream, a, tq, tiles);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_prefill_bf16(const PrefillArgs& a, int32_t head_dim, hipStream_t stream) {
  return head_dim == 128 ? launch_prefill_d<128>(a, stream) : launch_prefill_d<64>(a, stream);
}

}  // namespace pbb
