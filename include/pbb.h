/*
 * pbb.h -- C ABI of libpbb: Post-Boundary Bridge (PBB) decode attention on AMD Instinct
 * MI355X (gfx950), with a sliding-window (SWA) ring baseline built on the same kernels.
 *
 * Method (paper: "Post-Boundary Bridge: Must Local Attention Go Global Between Global
 * Layers?"):
 *   - A target at absolute position t sits in block p = B*floor(t/B) at phase r = t - p
 *     (Sec. 2.2, Eq.(1)).  Its PBB support is the causal block prefix {p..t}, plus the
 *     preceding half-block {p-h..p-1} when p > 0 and r < h, with h = B/2 (Sec. 3, Eq.(pbb)).
 *   - The output is one softmax over that support with scores q.k * scale, scale = 1/sqrt(d)
 *     by default (Sec. 3, Eq.(attention)); query head i reads KV head floor(i/G), G = Hq/Hkv
 *     (native grouped-query attention, Sec. 3 and Appendix F.1).
 *   - Keys and values live in a ring of B slots per (sequence, KV head): position s is stored
 *     at slot s mod B, so an append overwrites only a position that no current or future
 *     support needs and retained entries never move (Sec. 3 "Flash-PBB"; Appendix F.1,
 *     Proposition "Relocation-free PBB cache").
 *   - The SWA baseline attends over {max(0, t-W+1) .. t} (Prop. 2, Sec. 2.2) stored in a
 *     ring of S >= W slots (Appendix F.1 notes that a window can be kept in a ring as well).
 *
 * Layouts (row-major, contiguous, element type given by pbb_desc_t.dtype):
 *   q, out          [batch][n_q_heads][head_dim]
 *   k_new, v_new    [batch][n_kv_heads][head_dim]       key/value of the token at pos[b]
 *   k_ring, v_ring  [batch][n_kv_heads][slots][head_dim]
 *   pos             int32 [batch], 0 <= pos[b] < 2^31 - 1 (device memory)
 * Every pointer is DEVICE memory of the current HIP device and must be 16-byte aligned
 * (pos: 4-byte aligned).  A negative pos[b] makes that sequence's output zero and skips its
 * append.  Aliasing between any two buffers is undefined.
 *
 * Ownership: the caller allocates and frees every buffer, including the workspace.  The
 * library allocates nothing, keeps no pointer after a call returns, holds no global state
 * and is re-entrant.  Calls that take a stream only enqueue work on it (asynchronous); the
 * stream argument is a hipStream_t (NULL = the null stream).
 *
 * Errors: every entry point returns a pbb_status_t.  Arguments are checked on the host
 * before anything is enqueued; on any error nothing is launched and nothing is written.
 * No entry point aborts, prints, or lets a C++ exception escape.  PBB_ERR_LAUNCH reports a
 * failure returned by the HIP runtime when enqueueing.
 */
#ifndef PBB_H_
#define PBB_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PBB_OK = 0,
  PBB_ERR_NULL = 1,      /* a required pointer is NULL */
  PBB_ERR_SHAPE = 2,     /* inconsistent or unsupported sizes (see pbb_desc_t) */
  PBB_ERR_DTYPE = 3,     /* unsupported element type */
  PBB_ERR_ALIGN = 4,     /* a pointer is not 16-byte aligned (pos: 4-byte) */
  PBB_ERR_WORKSPACE = 5, /* workspace smaller than the size query returns */
  PBB_ERR_LAUNCH = 6     /* the HIP runtime refused the launch */
} pbb_status_t;

typedef enum {
  PBB_DTYPE_F32 = 0,  /* float32 inputs and outputs, float32 arithmetic throughout */
  PBB_DTYPE_BF16 = 1  /* bfloat16 inputs and outputs; fp32 accumulation; RNE on store */
} pbb_dtype_t;

/*
 * Problem description.  Constraints (PBB_ERR_SHAPE otherwise):
 *   batch >= 1; n_kv_heads >= 1; n_q_heads a multiple of n_kv_heads with
 *   G = n_q_heads / n_kv_heads <= 16; head_dim in {64, 128};
 *   PBB: block even, 2 <= block <= 65536, slots == block (the ring has exactly B slots);
 *   SWA: 1 <= window <= slots <= 65536 (block is ignored).
 * scale <= 0 selects 1/sqrt(head_dim) (Sec. 3, Eq.(attention)).
 * rope_base > 1 (bfloat16 decode only; PBB_ERR_DTYPE for float32): the decode step applies the
 * rotary position embedding itself (the paper's models use RoPE with base 10^6, Appendix C):
 * q and k_new are turned by their absolute position t before the scores, channel c < d/2
 * pairing with c + d/2 at angle t * rope_base^(-2c/d) (half-split pairs, as in the Qwen2.5
 * decoders the paper trains), rounded to bf16, and the turned key is what the ring receives,
 * so the ring holds rotated keys (slot mapping unchanged: positions stay absolute, Appendix
 * F.1).  v is not rotated.  Prefill takes already-rotated inputs and requires rope_base == 0.
 * rope_base == 0 leaves q and k_new as given; other values give PBB_ERR_SHAPE.
 */
typedef struct {
  int32_t batch;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t block;   /* PBB block size B; bridge width h = B/2 */
  int32_t window;  /* SWA window W (includes the current token); 0 for PBB */
  int32_t slots;   /* ring slots per (sequence, KV head) */
  int32_t dtype;   /* a pbb_dtype_t */
  float scale;
  float rope_base; /* 0: no rotary embedding; > 1: see below */
} pbb_desc_t;

/* Human-readable name of a status code (static storage; never NULL). */
const char *pbb_status_string(pbb_status_t status);

/*
 * Bytes of ONE ring tensor (K or V): batch * n_kv_heads * slots * head_dim * element size.
 * The paper's local KV storage, 2 * batch * B * H_KV * d_h * u, is twice this for the PBB
 * ring (Appendix F.1).  Validates desc as pbb_decode_step would (SWA rules when window > 0).
 */
pbb_status_t pbb_ring_bytes(const pbb_desc_t *desc, size_t *bytes_per_tensor);

/*
 * Enqueue zero-filling of both rings on `stream`.  A zeroed ring is the state before the
 * first decode step at position 0: for t < slots the support only covers positions that
 * have been appended (Appendix F.1, proof of the proposition).  The call is optional: the
 * decode steps never let a slot outside the support affect an output, whatever bits it holds
 * (NaN included), so rings may also start uninitialised or be loaded with pbb_ring_fill
 * with only the history the support needs.
 */
pbb_status_t pbb_ring_init(const pbb_desc_t *desc, void *k_ring, void *v_ring, void *stream);

/*
 * Enqueue a bulk load of history into the rings (the state a prefill leaves behind).
 * k_src, v_src: [batch][n_kv_heads][src_len][head_dim], row i holding absolute position
 * pos[b] - src_len + i of sequence b.  Each row with a non-negative position s is copied bit
 * for bit to slot s mod slots (Appendix F.1); rows with negative positions are skipped, as
 * are sequences with pos[b] < 0.  Requires 0 <= src_len <= slots.  pos is not modified: after
 * the call the rings hold exactly what sequential appends of those positions would leave.
 */
pbb_status_t pbb_ring_fill(const pbb_desc_t *desc, const int32_t *pos, const void *k_src,
                           const void *v_src, int32_t src_len, void *k_ring, void *v_ring,
                           void *stream);

/*
 * Workspace bytes pbb_decode_step needs.  0 unless the launch is split: bf16 launches with at
 * most 64 (sequence, KV head) units whose block (or window) exceeds 256 keys spread each unit's
 * support over S = min(floor(256 / units), ceil(steps / 8), 8) workgroups (steps = 32-key steps
 * of the longest support), which leave partial softmax states (Eq.(lse), Appendix A.4) in the
 * workspace for the last of them to merge.  Its first 256 bytes hold one counter per unit: they
 * must be zero-filled before the first call, and every call leaves them zero again, so one
 * allocation serves every later call on one stream, for any descriptor it is large enough for;
 * calls that may run concurrently need separate workspaces.  The size depends only on the
 * descriptor.
 */
pbb_status_t pbb_workspace_bytes(const pbb_desc_t *desc, size_t *bytes);

/*
 * One PBB decode step for every sequence, fused in a single kernel launch:
 *   1. append: k_ring[b][g][t mod B] <- k_new[b][g], same for V, t = pos[b]
 *      (Sec. 3 "Flash-PBB"; the overwritten position t - B is outside A(t), Appendix F.1);
 *   2. attention: out[b][i] = softmax over s in A_PBB(t) of (q[b][i] . k_s * scale) applied
 *      to v_s, for every query head i, with k_t, v_t taken from k_new, v_new
 *      (Eq.(pbb) with h = B/2, Eq.(attention)).
 * Requires slots == block and window ignored.  pos is read, never written: the caller
 * advances it (for example pos += 1 on the same stream) before the next step.
 * workspace: pbb_workspace_bytes bytes, 16-byte aligned, zero-filled before first use; may be
 * NULL when that is 0 (PBB_ERR_WORKSPACE if NULL or smaller otherwise).
 */
pbb_status_t pbb_decode_step(const pbb_desc_t *desc, const int32_t *pos, const void *q,
                             const void *k_new, const void *v_new, void *k_ring, void *v_ring,
                             void *out, void *workspace, size_t workspace_bytes, void *stream);

/* Workspace bytes swa_decode_step needs (the rules of pbb_workspace_bytes). */
pbb_status_t swa_workspace_bytes(const pbb_desc_t *desc, size_t *bytes);

/*
 * Sliding-window baseline with the same arguments: appends at slot t mod slots and attends
 * over {max(0, t-W+1) .. t} (Prop. 2), W = desc->window, read from a ring of desc->slots >= W
 * entries.  The overwritten position t - slots lies before the window, so no read races the
 * append.
 */
pbb_status_t swa_decode_step(const pbb_desc_t *desc, const int32_t *pos, const void *q,
                             const void *k_new, const void *v_new, void *k_ring, void *v_ring,
                             void *out, void *workspace, size_t workspace_bytes, void *stream);

/*
 * pbb_decode_step / swa_decode_step that also advance the positions on the device: the same
 * launch writes pos_next[b] = pos[b] + 1 (pos[b] itself when pos[b] < 0).  pos is not written,
 * and pos_next must not overlap pos (PBB_ERR_SHAPE), because other workgroups of the launch may
 * still be reading pos; a caller alternates two position buffers between steps.  This keeps a
 * step to a single kernel in captured graph sequences (the paper's decode runner advances
 * positions on the device, Appendix F.7).  pos_next: int32 [batch], 4-byte aligned.
 */
pbb_status_t pbb_decode_step_advance(const pbb_desc_t *desc, const int32_t *pos, int32_t *pos_next,
                                     const void *q, const void *k_new, const void *v_new,
                                     void *k_ring, void *v_ring, void *out, void *workspace,
                                     size_t workspace_bytes, void *stream);

pbb_status_t swa_decode_step_advance(const pbb_desc_t *desc, const int32_t *pos, int32_t *pos_next,
                                     const void *q, const void *k_new, const void *v_new,
                                     void *k_ring, void *v_ring, void *out, void *workspace,
                                     size_t workspace_bytes, void *stream);

/*
 * pbb_decode_step for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same step, with no
 * workspace argument.  When the launch needs a workspace (split launches: bf16, at most 64
 * (sequence, KV head) units, block above 256), it uses a buffer the library holds per device
 * -- PBB_NOALLOC_SCRATCH_BYTES bytes in a static device array, resolved on the first call on
 * each device (which also clears its counters with a fill kernel on `stream`, so a capture of
 * that first call records the clear) and kept until the process ends.  Never calls hipMalloc,
 * hipFree or an allocating routine.  Calls whose workspace would exceed that size return
 * PBB_ERR_WORKSPACE and enqueue nothing; every decode descriptor the library accepts fits.
 * Every call on one device shares the buffer and leaves its counters zero: calls that may
 * overlap on one GPU (other streams, other host threads) race and must be serialised by the
 * caller.  The stream must belong to the current HIP device.
 */
#define PBB_NOALLOC_SCRATCH_BYTES 4260096u
pbb_status_t pbb_decode_step_noalloc(const pbb_desc_t *desc, const int32_t *pos, const void *q,
                                     const void *k_new, const void *v_new, void *k_ring,
                                     void *v_ring, void *out, void *stream);

/*
 * Prefill: attention for every position of prompts at positions 0..n-1, the step that fills
 * the cache before decoding (Sec. 3: one fused kernel over block tiles and bridge rectangles
 * with log-sum-exp rescaling and native GQA; Appendix F.4: the added edges are h x h
 * target-by-source rectangles, no dense mask).  For every sequence b, position t < n and query
 * head i: out[b][t][i] = softmax over s in A_PBB(t) of (q[b][t][i] . k[b][s][floor(i/G)] *
 * scale) applied to v[b][s][floor(i/G)] (Eq.(pbb) with h = B/2, Eq.(attention)).
 *   q, out   [batch][n][n_q_heads][head_dim]   (token-major, as projections produce them)
 *   k, v     [batch][n][n_kv_heads][head_dim]
 *   lse      optional float32 [batch][n_q_heads][n]: log sum_{s in A(t)} e^{z_s}, natural log
 *            (the log-partition of Appendix A.4, Eq.(lse)); NULL skips it
 *   k_ring, v_ring  optional (both or neither), [batch][n_kv_heads][slots][head_dim]: every
 *            slot j that some position s in max(0, n - slots)..n-1 maps to (j = s mod slots)
 *            receives k/v of the last such s; other slots are left as they are.  After
 *            pbb_ring_init and this call, decoding continues with pos[b] = n (Appendix F.1).
 * bfloat16 only (PBB_ERR_DTYPE otherwise); fp32 accumulation, output rounded RNE.  Requires
 * 0 <= n <= 2^30 and n_q_heads * head_dim <= 2^24 (PBB_ERR_SHAPE otherwise); n == 0 does
 * nothing.  q, k, v, out, rings 16-byte aligned, lse 4-byte
 * aligned.  Same descriptor rules as pbb_decode_step, and rope_base must be 0 (rotate q and k
 * before the call; the ring then holds rotated keys as a rotary decode expects); no workspace.
 */
pbb_status_t pbb_prefill(const pbb_desc_t *desc, int32_t n, const void *q, const void *k,
                         const void *v, void *out, float *lse, void *k_ring, void *v_ring,
                         void *stream);

/* Sliding-window prefill with the same arguments: support {max(0, t-W+1) .. t} (Prop. 2),
 * W = desc->window, ring of desc->slots >= W entries (SWA descriptor rules). */
pbb_status_t swa_prefill(const pbb_desc_t *desc, int32_t n, const void *q, const void *k,
                         const void *v, void *out, float *lse, void *k_ring, void *v_ring,
                         void *stream);

/*
 * Training backward of the prefill attention: gradients with respect to q, k, v for an
 * upstream gradient dout of the prefill output (the paper's fused kernel includes backward
 * propagation, Sec. 3, and its grouped backward sums the query heads of a KV head, Appendix
 * F.4).  With p_s = exp(z_s - lse_t) over A(t) and delta_t = dout_t . out_t:
 *   dv_s += p_s dout_t,  dq_t = scale sum_s p_s (dout_t.v_s - delta_t) k_s,
 *   dk_s += scale p_s (dout_t.v_s - delta_t) q_t,
 * summed over the query heads of each KV head for dk and dv.
 *   q, out, dout, dq   [batch][n][n_q_heads][head_dim]   (out: the prefill output)
 *   k, v, dk, dv       [batch][n][n_kv_heads][head_dim]
 *   lse                float32 [batch][n_q_heads][n], the prefill's log-partitions
 * bfloat16 only; fp32 accumulation, gradients rounded RNE; every gradient element is written
 * once (no accumulation into the outputs; deterministic).  Requires rope_base == 0 (inputs
 * already rotated), 0 <= n <= 2^30 (n == 0 does nothing) and n_q_heads * head_dim <= 2^24
 * (PBB_ERR_SHAPE otherwise).  Alignment as pbb_prefill.
 * workspace: device memory of pbb_backward_workspace_bytes bytes = 8 * batch * n_q_heads * n
 * rounded up to a multiple of 256 (16-byte aligned, contents irrelevant; holds lse * log2(e)
 * and -delta per position); PBB_ERR_WORKSPACE if NULL or smaller.  Enqueues two kernels on
 * the stream.  The gradient buffers must not alias the inputs.
 */
pbb_status_t pbb_backward_workspace_bytes(const pbb_desc_t *desc, int32_t n, size_t *bytes);

pbb_status_t pbb_backward(const pbb_desc_t *desc, int32_t n, const void *q, const void *k,
                          const void *v, const void *out, const void *dout, const float *lse,
                          void *dq, void *dk, void *dv, void *workspace, size_t workspace_bytes,
                          void *stream);

/* Sliding-window counterpart of pbb_backward (support of Prop. 2; SWA descriptor rules). */
pbb_status_t swa_backward(const pbb_desc_t *desc, int32_t n, const void *q, const void *k,
                          const void *v, const void *out, const void *dout, const float *lse,
                          void *dq, void *dk, void *dv, void *workspace, size_t workspace_bytes,
                          void *stream);

#ifdef __cplusplus
}
#endif

#endif /* PBB_H_ */
