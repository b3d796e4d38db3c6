/*
 * Plain fp64 CPU oracle for Post-Boundary Bridge (PBB) decode attention.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or call this
 * file: only the test suite, the smoke check and the benchmark's CPU-baseline leg use it.
 * It shares no code, header or constant with the HIP library.
 *
 * What it computes (paper: "Post-Boundary Bridge: Must Local Attention Go Global
 * Between Global Layers?"):
 *   - block geometry p(t) = b*floor(t/b), r(t) = t - p(t)                 Sec. 2.2, Eq.(1)
 *   - the PBB support in its two-case form:                               Sec. 3, Eq.(pbb)
 *       A(t) = {p..t}  union  {p-h..p-1} if p > 0 and 0 <= r < h, else nothing
 *   - the sliding-window support {max(0,t-w+1)..t}                         Prop. 2 (Sec. 2.2)
 *   - single-softmax attention over a support, scores q.k/sqrt(d)          Sec. 3, Eq.(attention)
 *   - rotary positions (RoPE, base 10^6 in the paper's models), half-split pairs  Appendix C
 *   - backward: gradients of the prefill attention w.r.t. q, k, v        Sec. 3; App. F.4
 *   - prefill: every prompt position over its own support, with its log-partition
 *     log sum_s e^{z_s}                                                    Appendix A.4, Eq.(lse)
 * Keys and values are read from HISTORY arrays indexed by absolute position, never from
 * a ring, and every sum is taken in fp64 in plain position order.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

/* Membership of source s in the PBB support of target t (Eq.(pbb), two-case form). */
int oracle_pbb_member(int64_t t, int64_t s, int64_t block, int64_t bridge) {
    if (s < 0 || s > t) return 0;
    int64_t p = block * (t / block); /* block start, Eq.(1) */
    int64_t r = t - p;               /* target phase, Eq.(1) */
    if (s >= p) return 1;            /* causal block prefix {p..t} */
    if (p > 0 && r < bridge && s >= p - bridge && s <= p - 1) return 1; /* bridge */
    return 0;
}

/* Membership of source s in the sliding-window support of t (window includes t). */
int oracle_swa_member(int64_t t, int64_t s, int64_t window) {
    int64_t lo = t - window + 1;
    if (lo < 0) lo = 0;
    return s >= lo && s <= t;
}

/*
 * Unique-score counts over a length-n sequence (Appendix A.5, "Exact arithmetic matching"):
 * total = sum_t |A(t)|; cross = number of (t,s) pairs with s < p(t), i.e. sources in an
 * earlier block (block size `block` defines p).  Brute force over every (t, s) pair in a
 * window wide enough to hold the support; each membership is the definition above.
 */
void oracle_pbb_counts(int64_t n, int64_t block, int64_t bridge, int64_t *total, int64_t *cross) {
    int64_t tot = 0, cr = 0;
    for (int64_t t = 0; t < n; ++t) {
        int64_t p = block * (t / block);
        int64_t lo = p - bridge;
        if (lo < 0) lo = 0;
        for (int64_t s = lo; s <= t; ++s) {
            if (oracle_pbb_member(t, s, block, bridge)) {
                ++tot;
                if (s < p) ++cr;
            }
        }
    }
    *total = tot;
    *cross = cr;
}

void oracle_swa_counts(int64_t n, int64_t window, int64_t block, int64_t *total, int64_t *cross) {
    int64_t tot = 0, cr = 0;
    for (int64_t t = 0; t < n; ++t) {
        int64_t p = block * (t / block);
        int64_t lo = t - window;
        if (lo < 0) lo = 0;
        for (int64_t s = lo; s <= t; ++s) {
            if (oracle_swa_member(t, s, window)) {
                ++tot;
                if (s < p) ++cr;
            }
        }
    }
    *total = tot;
    *cross = cr;
}

/*
 * Single-softmax attention of one query over an explicit list of n keys (Eq.(attention)):
 *   z_s = scale * sum_c q[c] k[s][c];  o = sum_s e^{z_s} v_s / sum_s e^{z_s}.
 * The maximum score is subtracted before exponentiation (this changes no result).
 * Writes o[d] and, if lse != NULL, the log-partition log(sum_s e^{z_s}).
 * n == 0 writes zeros and lse = -inf (an empty support has Z = 0, Appendix A.4, Eq.(lse)).
 */
void oracle_attend(int64_t n, int64_t d, const double *q, const double *k, const double *v,
                   double scale, double *o, double *lse) {
    for (int64_t c = 0; c < d; ++c) o[c] = 0.0;
    if (n <= 0) {
        if (lse) *lse = -INFINITY;
        return;
    }
    double *z = (double *)malloc(sizeof(double) * (size_t)n);
    double m = -INFINITY;
    for (int64_t s = 0; s < n; ++s) {
        double acc = 0.0;
        for (int64_t c = 0; c < d; ++c) acc += q[c] * k[s * d + c];
        z[s] = acc * scale;
        if (z[s] > m) m = z[s];
    }
    double den = 0.0;
    for (int64_t s = 0; s < n; ++s) {
        double w = exp(z[s] - m);
        den += w;
        for (int64_t c = 0; c < d; ++c) o[c] += w * v[s * d + c];
    }
    for (int64_t c = 0; c < d; ++c) o[c] /= den;
    if (lse) *lse = m + log(den);
    free(z);
}

/*
 * Rotary position embedding of one head vector at absolute position `pos` (the models of the
 * paper use RoPE with base 10^6, Appendix C).  Half-split pairing, as in the Qwen2.5 decoders
 * the paper trains: channel c < d/2 pairs with c + d/2 and turns by the angle
 * pos * base^(-2c/d):
 *   out[c]       = x[c] cos(a) - x[c + d/2] sin(a)
 *   out[c + d/2] = x[c + d/2] cos(a) + x[c] sin(a)
 * Everything in fp64 (the angle itself is exact to ~1e-16 relative).
 */
static void rope_freqs(int64_t d, double base, double *freq) {
    for (int64_t c = 0; c < d / 2; ++c) freq[c] = pow(base, -2.0 * (double)c / (double)d);
}

static void rope_apply(int64_t d, int64_t pos, const double *freq, const double *x, double *out) {
    const int64_t half = d / 2;
    for (int64_t c = 0; c < half; ++c) {
        const double ang = (double)pos * freq[c];
        const double cs = cos(ang), sn = sin(ang);
        const double a = x[c], b = x[c + half];
        out[c] = a * cs - b * sn;
        out[c + half] = b * cs + a * sn;
    }
}

void oracle_rope(int64_t d, int64_t pos, double base, const double *x, double *out) {
    double *freq = (double *)malloc(sizeof(double) * (size_t)(d / 2 + 1));
    rope_freqs(d, base, freq);
    rope_apply(d, pos, freq, x, out);
    free(freq);
}

/* oracle_rope for n rows of float32 x [n][d], row r at position pos[r]; out [n][d] fp64. */
void oracle_rope_rows(int64_t d, int64_t n, const int64_t *pos, double base, const float *x,
                      double *out) {
    double *freq = (double *)malloc(sizeof(double) * (size_t)(d / 2 + 1));
    double *row = (double *)malloc(sizeof(double) * (size_t)d);
    rope_freqs(d, base, freq);
    for (int64_t r = 0; r < n; ++r) {
        for (int64_t c = 0; c < d; ++c) row[c] = (double)x[r * d + c];
        rope_apply(d, pos[r], freq, row, out + r * d);
    }
    free(row);
    free(freq);
}

/* ------------------------------------------------------------------------------------ */
/* Batched decode over absolute-position history.                                        */

typedef struct {
    int mode; /* 0 = PBB, 1 = SWA */
    int64_t batch, n_q_heads, n_kv_heads, head_dim, block, window;
    const int64_t *pos;
    const float *q;      /* [batch][Hq][d] */
    const float *k_hist; /* [batch][Hkv][hist_len][d], position s at row s - hist_lo[b] */
    const float *v_hist;
    const int64_t *hist_lo;
    int64_t hist_len;
    double scale;
    double rope_base; /* > 0: rotate q at t and every key at its own position (oracle_rope) */
    double *rope_freq; /* base^(-2c/d), c < d/2, when rope_base > 0 */
    double *out; /* [batch][Hq][d] */
    int64_t next;       /* next (b, head) work item */
    int error;
    pthread_mutex_t lock;
} decode_job;

static int member(const decode_job *j, int64_t t, int64_t s) {
    if (j->mode == 0) return oracle_pbb_member(t, s, j->block, j->block / 2);
    return oracle_swa_member(t, s, j->window);
}

static void decode_one(decode_job *j, int64_t item, double *z, double *qd) {
    const int64_t d = j->head_dim;
    const int64_t G = j->n_q_heads / j->n_kv_heads;
    const int64_t b = item / j->n_q_heads, i = item % j->n_q_heads;
    const int64_t g = i / G; /* query head i reads KV head floor(i/G) */
    const int64_t t = j->pos[b];
    double *o = j->out + (b * j->n_q_heads + i) * d;
    for (int64_t c = 0; c < d; ++c) o[c] = 0.0;
    if (t < 0) return;
    for (int64_t c = 0; c < d; ++c) qd[c] = (double)j->q[(b * j->n_q_heads + i) * d + c];
    double *kr = qd + d; /* scratch: one rotated key row, then the raw row */
    double *kraw = qd + 2 * d;
    if (j->rope_base > 0.0) {
        for (int64_t c = 0; c < d; ++c) kraw[c] = qd[c];
        rope_apply(d, t, j->rope_freq, kraw, qd);
    }
    /* Candidate window: wide enough to contain every source either definition admits. */
    int64_t span = (j->mode == 0) ? (j->block + j->block / 2) : j->window;
    int64_t lo = t - span;
    if (lo < 0) lo = 0;
    const float *kh = j->k_hist + (b * j->n_kv_heads + g) * j->hist_len * d;
    const float *vh = j->v_hist + (b * j->n_kv_heads + g) * j->hist_len * d;
    double m = -INFINITY;
    int64_t cnt = 0;
    for (int64_t s = lo; s <= t; ++s) {
        if (!member(j, t, s)) continue;
        int64_t row = s - j->hist_lo[b];
        if (row < 0 || row >= j->hist_len) {
            j->error = 1; /* the caller did not supply this history position */
            return;
        }
        double acc = 0.0;
        if (j->rope_base > 0.0) {
            for (int64_t c = 0; c < d; ++c) kraw[c] = (double)kh[row * d + c];
            rope_apply(d, s, j->rope_freq, kraw, kr);
            for (int64_t c = 0; c < d; ++c) acc += qd[c] * kr[c];
        } else {
            for (int64_t c = 0; c < d; ++c) acc += qd[c] * (double)kh[row * d + c];
        }
        z[s - lo] = acc * j->scale;
        if (z[s - lo] > m) m = z[s - lo];
        ++cnt;
    }
    double den = 0.0;
    for (int64_t s = lo; s <= t; ++s) {
        if (!member(j, t, s)) continue;
        int64_t row = s - j->hist_lo[b];
        double w = exp(z[s - lo] - m);
        den += w;
        for (int64_t c = 0; c < d; ++c) o[c] += w * (double)vh[row * d + c];
    }
    (void)cnt;
    for (int64_t c = 0; c < d; ++c) o[c] /= den;
}

static void *decode_worker(void *arg) {
    decode_job *j = (decode_job *)arg;
    int64_t span = (j->mode == 0) ? (j->block + j->block / 2) : j->window;
    double *z = (double *)malloc(sizeof(double) * (size_t)(span + 1));
    double *qd = (double *)malloc(sizeof(double) * (size_t)(3 * j->head_dim));
    const int64_t total = j->batch * j->n_q_heads;
    for (;;) {
        pthread_mutex_lock(&j->lock);
        int64_t item = j->next;
        j->next += 1;
        pthread_mutex_unlock(&j->lock);
        if (item >= total) break;
        decode_one(j, item, z, qd);
    }
    free(z);
    free(qd);
    return NULL;
}

/*
 * One decode step for a batch: for every sequence b and query head i, attention of
 * q[b][i] over the support of t = pos[b] (PBB with h = block/2 when mode == 0, SWA with
 * the given window when mode == 1).  Returns 0 on success, 1 if some needed history
 * position lies outside [hist_lo[b], hist_lo[b] + hist_len), 2 on bad arguments.
 * n_threads <= 0 uses every online core.
 */
static int decode_run(int mode, int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                      int64_t head_dim, int64_t block, int64_t window, const int64_t *pos,
                      const float *q, const float *k_hist, const float *v_hist,
                      const int64_t *hist_lo, int64_t hist_len, double scale, double rope_base,
                      double *out, int n_threads);

int oracle_decode(int mode, int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                  int64_t head_dim, int64_t block, int64_t window, const int64_t *pos,
                  const float *q, const float *k_hist, const float *v_hist,
                  const int64_t *hist_lo, int64_t hist_len, double scale, double *out,
                  int n_threads) {
    return decode_run(mode, batch, n_q_heads, n_kv_heads, head_dim, block, window, pos, q,
                      k_hist, v_hist, hist_lo, hist_len, scale, 0.0, out, n_threads);
}

/*
 * oracle_decode with rotary positions: q at its position t and every history key at its own
 * absolute position s are rotated by oracle_rope (base rope_base > 0) before the scores; the
 * history holds unrotated keys, values are not rotated.
 */
int oracle_decode_rope(int mode, int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                       int64_t head_dim, int64_t block, int64_t window, const int64_t *pos,
                       const float *q, const float *k_hist, const float *v_hist,
                       const int64_t *hist_lo, int64_t hist_len, double scale, double rope_base,
                       double *out, int n_threads) {
    if (!(rope_base > 1.0) || head_dim % 2 != 0) return 2;
    return decode_run(mode, batch, n_q_heads, n_kv_heads, head_dim, block, window, pos, q,
                      k_hist, v_hist, hist_lo, hist_len, scale, rope_base, out, n_threads);
}

static int decode_run(int mode, int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                      int64_t head_dim, int64_t block, int64_t window, const int64_t *pos,
                      const float *q, const float *k_hist, const float *v_hist,
                      const int64_t *hist_lo, int64_t hist_len, double scale, double rope_base,
                      double *out, int n_threads) {
    if (batch < 0 || n_q_heads <= 0 || n_kv_heads <= 0 || head_dim <= 0) return 2;
    if (n_q_heads % n_kv_heads != 0) return 2;
    if (mode == 0 && (block < 2 || block % 2 != 0)) return 2;
    if (mode == 1 && window < 1) return 2;
    decode_job j;
    memset(&j, 0, sizeof(j));
    j.mode = mode;
    j.batch = batch;
    j.n_q_heads = n_q_heads;
    j.n_kv_heads = n_kv_heads;
    j.head_dim = head_dim;
    j.block = block;
    j.window = window;
    j.pos = pos;
    j.q = q;
    j.k_hist = k_hist;
    j.v_hist = v_hist;
    j.hist_lo = hist_lo;
    j.hist_len = hist_len;
    j.scale = scale;
    j.rope_base = rope_base;
    j.rope_freq = NULL;
    if (rope_base > 0.0) {
        j.rope_freq = (double *)malloc(sizeof(double) * (size_t)(head_dim / 2 + 1));
        rope_freqs(head_dim, rope_base, j.rope_freq);
    }
    j.out = out;
    pthread_mutex_init(&j.lock, NULL);
    if (n_threads <= 0) n_threads = (int)sysconf(_SC_NPROCESSORS_ONLN);
    if (n_threads < 1) n_threads = 1;
    if (n_threads > 256) n_threads = 256;
    pthread_t th[256];
    for (int i = 0; i < n_threads; ++i) pthread_create(&th[i], NULL, decode_worker, &j);
    for (int i = 0; i < n_threads; ++i) pthread_join(th[i], NULL);
    pthread_mutex_destroy(&j.lock);
    free(j.rope_freq);
    return j.error ? 1 : 0;
}

/* ------------------------------------------------------------------------------------ */
/* Prefill: every position of a prompt attends over its own support.                     */

typedef struct {
    int mode; /* 0 = PBB, 1 = SWA */
    int64_t batch, n, n_q_heads, n_kv_heads, head_dim, block, window;
    const float *q; /* [batch][n][Hq][d] */
    const float *k; /* [batch][n][Hkv][d], position s of sequence b at row s */
    const float *v;
    double scale;
    double *out; /* [batch][n][Hq][d] */
    double *lse; /* [batch][Hq][n] */
    int64_t next;
    pthread_mutex_t lock;
} prefill_job;

static int prefill_member(const prefill_job *j, int64_t t, int64_t s) {
    if (j->mode == 0) return oracle_pbb_member(t, s, j->block, j->block / 2);
    return oracle_swa_member(t, s, j->window);
}

/* One (sequence, position, query head): scores over the support in position order, then
 * o = sum_s e^{z_s - m} v_s / sum_s e^{z_s - m} and lse = m + log sum_s e^{z_s - m}. */
static void prefill_one(prefill_job *j, int64_t item, double *z, double *qd) {
    const int64_t d = j->head_dim, hq = j->n_q_heads, hkv = j->n_kv_heads, n = j->n;
    const int64_t G = hq / hkv;
    const int64_t i = item % hq;
    const int64_t t = (item / hq) % n;
    const int64_t b = item / (hq * n);
    const int64_t g = i / G; /* query head i reads KV head floor(i/G) */
    double *o = j->out + ((b * n + t) * hq + i) * d;
    for (int64_t c = 0; c < d; ++c) {
        o[c] = 0.0;
        qd[c] = (double)j->q[((b * n + t) * hq + i) * d + c];
    }
    const int64_t span = (j->mode == 0) ? (j->block + j->block / 2) : j->window;
    int64_t lo = t - span;
    if (lo < 0) lo = 0;
    double m = -INFINITY;
    for (int64_t s = lo; s <= t; ++s) {
        if (!prefill_member(j, t, s)) continue;
        const float *ks = j->k + ((b * n + s) * hkv + g) * d;
        double acc = 0.0;
        for (int64_t c = 0; c < d; ++c) acc += qd[c] * (double)ks[c];
        z[s - lo] = acc * j->scale;
        if (z[s - lo] > m) m = z[s - lo];
    }
    double den = 0.0;
    for (int64_t s = lo; s <= t; ++s) {
        if (!prefill_member(j, t, s)) continue;
        const float *vs = j->v + ((b * n + s) * hkv + g) * d;
        double w = exp(z[s - lo] - m);
        den += w;
        for (int64_t c = 0; c < d; ++c) o[c] += w * (double)vs[c];
    }
    for (int64_t c = 0; c < d; ++c) o[c] /= den;
    j->lse[(b * hq + i) * n + t] = m + log(den);
}

static void *prefill_worker(void *arg) {
    prefill_job *j = (prefill_job *)arg;
    int64_t span = (j->mode == 0) ? (j->block + j->block / 2) : j->window;
    double *z = (double *)malloc(sizeof(double) * (size_t)(span + 1));
    double *qd = (double *)malloc(sizeof(double) * (size_t)j->head_dim);
    const int64_t total = j->batch * j->n * j->n_q_heads;
    for (;;) {
        pthread_mutex_lock(&j->lock);
        int64_t first = j->next;
        j->next += 64;
        pthread_mutex_unlock(&j->lock);
        if (first >= total) break;
        int64_t last = first + 64 < total ? first + 64 : total;
        for (int64_t item = first; item < last; ++item) prefill_one(j, item, z, qd);
    }
    free(z);
    free(qd);
    return NULL;
}

/*
 * Prefill of a batch of prompts of n tokens at positions 0..n-1: for every sequence b,
 * position t and query head i, attention of q[b][t][i] over the support of t (PBB with
 * h = block/2 when mode == 0, Eq.(pbb); SWA with the given window when mode == 1, Prop. 2),
 * Eq.(attention), plus the log-partition lse = log sum_{s in A(t)} e^{z_s} (Appendix A.4,
 * Eq.(lse)).  Layouts: q, out [batch][n][Hq][d]; k, v [batch][n][Hkv][d]; lse [batch][Hq][n].
 * Returns 0 on success, 2 on bad arguments.  n_threads <= 0 uses every online core.
 */
int oracle_prefill(int mode, int64_t batch, int64_t n, int64_t n_q_heads, int64_t n_kv_heads,
                   int64_t head_dim, int64_t block, int64_t window, const float *q,
                   const float *k, const float *v, double scale, double *out, double *lse,
                   int n_threads) {
    if (batch < 0 || n < 0 || n_q_heads <= 0 || n_kv_heads <= 0 || head_dim <= 0) return 2;
    if (n_q_heads % n_kv_heads != 0) return 2;
    if (mode == 0 && (block < 2 || block % 2 != 0)) return 2;
    if (mode == 1 && window < 1) return 2;
    prefill_job j;
    memset(&j, 0, sizeof(j));
    j.mode = mode;
    j.batch = batch;
    j.n = n;
    j.n_q_heads = n_q_heads;
    j.n_kv_heads = n_kv_heads;
    j.head_dim = head_dim;
    j.block = block;
    j.window = window;
    j.q = q;
    j.k = k;
    j.v = v;
    j.scale = scale;
    j.out = out;
    j.lse = lse;
    pthread_mutex_init(&j.lock, NULL);
    if (n_threads <= 0) n_threads = (int)sysconf(_SC_NPROCESSORS_ONLN);
    if (n_threads < 1) n_threads = 1;
    if (n_threads > 256) n_threads = 256;
    pthread_t th[256];
    for (int i = 0; i < n_threads; ++i) pthread_create(&th[i], NULL, prefill_worker, &j);
    for (int i = 0; i < n_threads; ++i) pthread_join(th[i], NULL);
    pthread_mutex_destroy(&j.lock);
    return 0;
}

/* ------------------------------------------------------------------------------------ */
/* Backward of the prefill attention (training): gradients of q, k, v.                   */

typedef struct {
    int mode;
    int64_t batch, n, n_q_heads, n_kv_heads, head_dim, block, window;
    const float *q, *k, *v, *dout; /* q, dout [batch][n][Hq][d]; k, v [batch][n][Hkv][d] */
    double scale;
    double *dq, *dk, *dv; /* dq [batch][n][Hq][d]; dk, dv [batch][n][Hkv][d] */
    int64_t next;
    pthread_mutex_t lock;
} backward_job;

static int backward_member(const backward_job *j, int64_t t, int64_t s) {
    if (j->mode == 0) return oracle_pbb_member(t, s, j->block, j->block / 2);
    return oracle_swa_member(t, s, j->window);
}

/*
 * All query heads of one (sequence, KV head) pair, every position t.  With o = sum_s p_s v_s,
 * p_s = e^{z_s} / sum_u e^{z_u}, z_s = scale q.k_s over the support A(t) (Eq.(attention)) and an
 * upstream gradient g = dL/do:
 *   dL/dv_s += p_s g;   dL/dp_s = g.v_s;   dL/dz_s = p_s (g.v_s - g.o);
 *   dL/dq += scale sum_s dL/dz_s k_s;   dL/dk_s += scale dL/dz_s q.
 * Query heads of the KV head add into the same dk, dv (grouped-query attention).
 */
static void backward_one(backward_job *j, int64_t item, double *z, double *o, double *qd,
                         double *gd) {
    const int64_t d = j->head_dim, hq = j->n_q_heads, hkv = j->n_kv_heads, n = j->n;
    const int64_t G = hq / hkv;
    const int64_t b = item / hkv, g = item % hkv;
    const int64_t span = (j->mode == 0) ? (j->block + j->block / 2) : j->window;
    for (int64_t i = g * G; i < (g + 1) * G; ++i) {
        for (int64_t t = 0; t < n; ++t) {
            int64_t lo = t - span;
            if (lo < 0) lo = 0;
            for (int64_t c = 0; c < d; ++c) {
                qd[c] = (double)j->q[((b * n + t) * hq + i) * d + c];
                gd[c] = (double)j->dout[((b * n + t) * hq + i) * d + c];
                o[c] = 0.0;
            }
            double m = -INFINITY;
            for (int64_t s = lo; s <= t; ++s) {
                if (!backward_member(j, t, s)) continue;
                const float *ks = j->k + ((b * n + s) * hkv + g) * d;
                double acc = 0.0;
                for (int64_t c = 0; c < d; ++c) acc += qd[c] * (double)ks[c];
                z[s - lo] = acc * j->scale;
                if (z[s - lo] > m) m = z[s - lo];
            }
            double den = 0.0;
            for (int64_t s = lo; s <= t; ++s) {
                if (!backward_member(j, t, s)) continue;
                z[s - lo] = exp(z[s - lo] - m);
                den += z[s - lo];
            }
            for (int64_t s = lo; s <= t; ++s) {
                if (!backward_member(j, t, s)) continue;
                z[s - lo] /= den; /* p_s */
                const float *vs = j->v + ((b * n + s) * hkv + g) * d;
                for (int64_t c = 0; c < d; ++c) o[c] += z[s - lo] * (double)vs[c];
            }
            double go = 0.0;
            for (int64_t c = 0; c < d; ++c) go += gd[c] * o[c];
            double *dqt = j->dq + ((b * n + t) * hq + i) * d;
            for (int64_t s = lo; s <= t; ++s) {
                if (!backward_member(j, t, s)) continue;
                const double p = z[s - lo];
                const float *ks = j->k + ((b * n + s) * hkv + g) * d;
                const float *vs = j->v + ((b * n + s) * hkv + g) * d;
                double gv = 0.0;
                for (int64_t c = 0; c < d; ++c) gv += gd[c] * (double)vs[c];
                const double dz = p * (gv - go);
                double *dks = j->dk + ((b * n + s) * hkv + g) * d;
                double *dvs = j->dv + ((b * n + s) * hkv + g) * d;
                for (int64_t c = 0; c < d; ++c) {
                    dvs[c] += p * gd[c];
                    dqt[c] += j->scale * dz * (double)ks[c];
                    dks[c] += j->scale * dz * qd[c];
                }
            }
        }
    }
}

static void *backward_worker(void *arg) {
    backward_job *j = (backward_job *)arg;
    const int64_t span = (j->mode == 0) ? (j->block + j->block / 2) : j->window;
    double *z = (double *)malloc(sizeof(double) * (size_t)(span + 1));
    double *buf = (double *)malloc(sizeof(double) * (size_t)(3 * j->head_dim));
    const int64_t total = j->batch * j->n_kv_heads;
    for (;;) {
        pthread_mutex_lock(&j->lock);
        int64_t item = j->next;
        j->next += 1;
        pthread_mutex_unlock(&j->lock);
        if (item >= total) break;
        backward_one(j, item, z, buf, buf + j->head_dim, buf + 2 * j->head_dim);
    }
    free(z);
    free(buf);
    return NULL;
}

/*
 * Gradients of the prefill attention (positions 0..n-1, support Eq.(pbb) with h = block/2 when
 * mode == 0, Prop. 2 when mode == 1) for an upstream gradient dout of the output: dq, dk, dv in
 * fp64, zero-initialised here.  Layouts as oracle_prefill; dk, dv [batch][n][Hkv][d].
 * Returns 0, or 2 on bad arguments.
 */
int oracle_backward(int mode, int64_t batch, int64_t n, int64_t n_q_heads, int64_t n_kv_heads,
                    int64_t head_dim, int64_t block, int64_t window, const float *q,
                    const float *k, const float *v, const float *dout, double scale, double *dq,
                    double *dk, double *dv, int n_threads) {
    if (batch < 0 || n < 0 || n_q_heads <= 0 || n_kv_heads <= 0 || head_dim <= 0) return 2;
    if (n_q_heads % n_kv_heads != 0) return 2;
    if (mode == 0 && (block < 2 || block % 2 != 0)) return 2;
    if (mode == 1 && window < 1) return 2;
    memset(dq, 0, sizeof(double) * (size_t)(batch * n * n_q_heads * head_dim));
    memset(dk, 0, sizeof(double) * (size_t)(batch * n * n_kv_heads * head_dim));
    memset(dv, 0, sizeof(double) * (size_t)(batch * n * n_kv_heads * head_dim));
    backward_job j;
    memset(&j, 0, sizeof(j));
    j.mode = mode;
    j.batch = batch;
    j.n = n;
    j.n_q_heads = n_q_heads;
    j.n_kv_heads = n_kv_heads;
    j.head_dim = head_dim;
    j.block = block;
    j.window = window;
    j.q = q;
    j.k = k;
    j.v = v;
    j.dout = dout;
    j.scale = scale;
    j.dq = dq;
    j.dk = dk;
    j.dv = dv;
    pthread_mutex_init(&j.lock, NULL);
    if (n_threads <= 0) n_threads = (int)sysconf(_SC_NPROCESSORS_ONLN);
    if (n_threads < 1) n_threads = 1;
    if (n_threads > 256) n_threads = 256;
    pthread_t th[256];
    for (int i = 0; i < n_threads; ++i) pthread_create(&th[i], NULL, backward_worker, &j);
    for (int i = 0; i < n_threads; ++i) pthread_join(th[i], NULL);
    pthread_mutex_destroy(&j.lock);
    return 0;
}
