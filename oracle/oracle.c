/*
 * oracle.c -- plain fp64 CPU reference for MagicDec's two attention calls.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or
 * calls this file: only tests/, __graft_entry__.smoke() and the cpu_baseline
 * leg of bench.py may.  It shares no header, helper, table or kernel with the
 * GPU library.
 *
 * What it computes (MagicDec, arXiv 2408.11049):
 *   - Verification (Sec. 3.1, T_V(B,S,gamma); Sec. 3.2, verify and decode
 *     share the KV loading): the gamma+1 speculated query tokens of each
 *     sequence attend to the full KV cache, causally among themselves.
 *   - Drafting with a StreamingLLM-style sparse KV (Sec. 4.1, Eq. 3 budget K;
 *     Sec. 5.1 setup, StreamingLLM-style draft cache): each query attends to
 *     the sink tokens plus a window of its most recent tokens.
 *   - Drafting with a static compressed cache given as token positions
 *     (SnapKV-style selection made at prefill; Sec. 4.4, Sec. 5.2): each
 *     query attends to the listed prompt positions plus the speculated
 *     tokens, causally.
 *   - The log-sum-exp merge of attention computed over disjoint key sets
 *     (the Flash-Decoding split-KV identity named in Sec. 2).
 *
 * Readings where the paper is silent (each listed in the design notes):
 *   - q_len = gamma+1 query rows per sequence (Eq. 1 counts gamma+1 tokens).
 *   - kv_lens[b] already counts the q_len new tokens; query i of sequence b
 *     sits at position p = kv_lens[b] - q_len + i (bottom-right alignment).
 *   - Draft key set for the query at position p:
 *       { j <= p : j < n_sink  or  j >= p - window + 1 }.
 *   - Indexed draft key set of sequence b, kv head hk: the listed positions
 *     idx[b][hk][0 .. idx_len[b]) that lie in [0, S - q_len), taken as a set,
 *     plus the speculated positions S - q_len .. p.
 *   - GQA: query head h reads kv head h / (Hq / Hkv).
 *   - Scale: the caller's scale (default 1/sqrt(d)); lse in natural log.
 *
 * The softmax is the direct two-pass definition: all scores of the row are
 * formed, the maximum is subtracted, exponentials are summed, then
 * O = sum_j e_j V_j / Z and lse = m + ln Z.  No online rescaling, no tiling.
 * All arithmetic is in double; bf16 and fp32 inputs convert exactly.
 *
 * Threads (pthreads) only split independent (b, i, h) rows.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_F32 0
#define ORACLE_BF16 1
#define ORACLE_VERIFY 0
#define ORACLE_DRAFT 1
#define ORACLE_INDEXED 2

/* A bf16 value is the upper 16 bits of the fp32 with the same sign,
 * exponent and leading 7 mantissa bits, so widening is exact. */
static double load_elem(const void* base, int dtype, int64_t idx) {
  if (dtype == ORACLE_F32) return (double)((const float*)base)[idx];
  uint32_t bits = ((uint32_t)((const uint16_t*)base)[idx]) << 16;
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

typedef struct {
  int mode, B, q_len, Hq, Hkv, d, dtype;
  double scale;
  const void *q, *k, *v;
  int64_t s_blk, s_tok, s_head;
  int page_size;
  const int32_t* page_table;
  int max_pages;
  const int32_t* kv_lens;
  int n_sink, window;
  double* o;
  double* lse;
  double* probs;
  int probs_len;
  const int32_t* idx;     /* indexed mode: [B][Hkv][idx_stride] positions */
  const int32_t* idx_len; /* indexed mode: [B] list lengths */
  int idx_stride;
  int nthreads, tid;
  int status;
} job_t;

/* Element offset of (token j, kv head hk, channel 0) of sequence b. */
static int64_t kv_offset(const job_t* a, int b, int j, int hk) {
  int64_t blk, tok;
  if (a->page_size == 0) {
    blk = b;
    tok = j;
  } else {
    blk = a->page_table[(int64_t)b * a->max_pages + j / a->page_size];
    tok = j % a->page_size;
  }
  return blk * a->s_blk + tok * a->s_tok + (int64_t)hk * a->s_head;
}

/* Is key j visible to the query at position p?  member: indexed mode only,
 * member[j] != 0 iff j is a listed prompt position of this (b, kv head). */
static int visible(const job_t* a, int j, int p, int S, const unsigned char* member) {
  if (j > p) return 0;
  if (a->mode == ORACLE_VERIFY) return 1;
  if (a->mode == ORACLE_INDEXED) return j >= S - a->q_len || member[j];
  return j < a->n_sink || j >= p - a->window + 1;
}

static void* run_rows(void* arg) {
  job_t* a = (job_t*)arg;
  int G = a->Hq / a->Hkv;
  int64_t n_rows = (int64_t)a->B * a->q_len * a->Hq;
  int S_cap = 0;
  for (int b = 0; b < a->B; ++b)
    if (a->kv_lens[b] > S_cap) S_cap = a->kv_lens[b];
  double* score = (double*)malloc(sizeof(double) * (size_t)(S_cap > 0 ? S_cap : 1));
  double* acc = (double*)malloc(sizeof(double) * (size_t)a->d);
  unsigned char* member = (unsigned char*)malloc((size_t)(S_cap > 0 ? S_cap : 1));
  if (!score || !acc || !member) {
    a->status = -1;
    free(score);
    free(acc);
    free(member);
    return NULL;
  }
  for (int64_t row = a->tid; row < n_rows; row += a->nthreads) {
    /* row = (b * q_len + i) * Hq + h, the order of the output tensor. */
    int h = (int)(row % a->Hq);
    int i = (int)((row / a->Hq) % a->q_len);
    int b = (int)(row / ((int64_t)a->Hq * a->q_len));
    int hk = h / G;
    int S = a->kv_lens[b];
    int p = S - a->q_len + i;
    const int64_t q_off = row * a->d;
    if (a->mode == ORACLE_INDEXED) {
      /* The list as a set of prompt positions; anything outside [0, S - q_len) is ignored. */
      memset(member, 0, (size_t)(S > 0 ? S : 1));
      const int32_t* list = a->idx + ((int64_t)b * a->Hkv + hk) * a->idx_stride;
      int n = a->idx_len[b] < a->idx_stride ? a->idx_len[b] : a->idx_stride;
      for (int t = 0; t < n; ++t)
        if (list[t] >= 0 && list[t] < S - a->q_len) member[list[t]] = 1;
    }

    /* Pass 1: scores of every visible key, and their maximum. */
    double m = -INFINITY;
    for (int j = 0; j < S; ++j) {
      if (!visible(a, j, p, S, member)) continue;
      int64_t k_off = kv_offset(a, b, j, hk);
      double dot = 0.0;
      for (int c = 0; c < a->d; ++c)
        dot += load_elem(a->q, a->dtype, q_off + c) * load_elem(a->k, a->dtype, k_off + c);
      score[j] = a->scale * dot;
      if (score[j] > m) m = score[j];
    }
    /* Pass 2: Z = sum exp(s - m), O = sum exp(s - m) V / Z. */
    double Z = 0.0;
    for (int c = 0; c < a->d; ++c) acc[c] = 0.0;
    for (int j = 0; j < S; ++j) {
      if (!visible(a, j, p, S, member)) continue;
      double e = exp(score[j] - m);
      Z += e;
      int64_t v_off = kv_offset(a, b, j, hk);
      for (int c = 0; c < a->d; ++c) acc[c] += e * load_elem(a->v, a->dtype, v_off + c);
    }
    for (int c = 0; c < a->d; ++c) a->o[row * a->d + c] = Z > 0.0 ? acc[c] / Z : 0.0;
    if (a->lse) a->lse[row] = Z > 0.0 ? m + log(Z) : -INFINITY;
    if (a->probs) {
      double* pr = a->probs + row * a->probs_len;
      for (int j = 0; j < a->probs_len; ++j) pr[j] = 0.0;
      for (int j = 0; j < S && j < a->probs_len; ++j)
        if (visible(a, j, p, S, member)) pr[j] = exp(score[j] - m) / Z;
    }
  }
  free(score);
  free(acc);
  free(member);
  return NULL;
}

/*
 * oracle_attention: O[b, i, h, :] and lse[b, i, h] for every row.
 *   q        [B, q_len, Hq, d]
 *   k, v     element (b or page, token-in-block, kv head, channel) at
 *            blk * s_blk + tok * s_tok + hk * s_head + c
 *   page_size 0 = contiguous (blk = b, tok = j); otherwise the block of key j
 *            is page_table[b * max_pages + j / page_size], tok = j % page_size
 *   o        [B, q_len, Hq, d] double;  lse [B, q_len, Hq] double or NULL
 *   probs    NULL, or [B, q_len, Hq, probs_len] explicit softmax rows
 * Returns 0 on success, -1 on a bad argument or allocation failure.
 */
static int run_all(job_t base);

int oracle_attention(int mode, int B, int q_len, int Hq, int Hkv, int d, int dtype, double scale,
                     const void* q, const void* k, const void* v, int64_t s_blk, int64_t s_tok,
                     int64_t s_head, int page_size, const int32_t* page_table, int max_pages,
                     const int32_t* kv_lens, int n_sink, int window, double* o, double* lse,
                     double* probs, int probs_len, int nthreads) {
  if (mode != ORACLE_VERIFY && mode != ORACLE_DRAFT) return -1;
  if (mode == ORACLE_DRAFT && (n_sink < 0 || window < 1)) return -1;
  job_t base = {mode, B, q_len, Hq, Hkv, d, dtype, scale, q, k, v, s_blk, s_tok, s_head,
                page_size, page_table, max_pages, kv_lens, n_sink, window, o, lse, probs,
                probs_len, NULL, NULL, 0, nthreads, 0, 0};
  return run_all(base);
}

/*
 * oracle_attention_indexed: draft attention over a listed static cache.
 *   idx     [B][Hkv][idx_stride] int32 prompt positions, any order, unique
 *   idx_len [B] int32, entries beyond it (or idx_stride) are ignored
 * Other arguments as oracle_attention.
 */
int oracle_attention_indexed(int B, int q_len, int Hq, int Hkv, int d, int dtype, double scale,
                             const void* q, const void* k, const void* v, int64_t s_blk,
                             int64_t s_tok, int64_t s_head, int page_size,
                             const int32_t* page_table, int max_pages, const int32_t* kv_lens,
                             const int32_t* idx, const int32_t* idx_len, int idx_stride,
                             double* o, double* lse, double* probs, int probs_len, int nthreads) {
  if (idx_stride < 0 || (B > 0 && idx_stride > 0 && (!idx || !idx_len))) return -1;
  if (B > 0 && !idx_len) return -1;
  job_t base = {ORACLE_INDEXED, B, q_len, Hq, Hkv, d, dtype, scale, q, k, v, s_blk, s_tok,
                s_head, page_size, page_table, max_pages, kv_lens, 0, 1, o, lse, probs,
                probs_len, idx, idx_len, idx_stride, nthreads, 0, 0};
  return run_all(base);
}

static int run_all(job_t base) {
  const int B = base.B, q_len = base.q_len, Hq = base.Hq, Hkv = base.Hkv, d = base.d;
  if (B < 0 || q_len < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || d < 1) return -1;
  if (base.dtype != ORACLE_F32 && base.dtype != ORACLE_BF16) return -1;
  if (base.page_size < 0 || (base.page_size > 0 && !base.page_table)) return -1;
  if (B == 0) return 0;
  if (!base.q || !base.k || !base.v || !base.o || !base.kv_lens) return -1;
  int nthreads = base.nthreads < 1 ? 1 : base.nthreads;
  base.nthreads = nthreads;
  job_t* jobs = (job_t*)malloc(sizeof(job_t) * (size_t)nthreads);
  pthread_t* th = (pthread_t*)malloc(sizeof(pthread_t) * (size_t)nthreads);
  if (!jobs || !th) {
    free(jobs);
    free(th);
    return -1;
  }
  for (int t = 0; t < nthreads; ++t) {
    jobs[t] = base;
    jobs[t].tid = t;
  }
  int started = 0;
  for (int t = 1; t < nthreads; ++t) {
    if (pthread_create(&th[t], NULL, run_rows, &jobs[t]) != 0) break;
    started = t;
  }
  run_rows(&jobs[0]);
  for (int t = started + 1; t < nthreads; ++t) run_rows(&jobs[t]); /* threads that failed to start */
  for (int t = 1; t <= started; ++t) pthread_join(th[t], NULL);
  int status = 0;
  for (int t = 0; t < nthreads; ++t)
    if (jobs[t].status) status = -1;
  free(jobs);
  free(th);
  return status;
}

/*
 * oracle_merge_lse: combine attention results computed over disjoint key
 * sets.  For every row:  lse = ln sum_k exp(lse_k),
 *                        O   = sum_k exp(lse_k - lse) O_k.
 * Parts with lse_k = -inf contribute nothing; if every part is empty the row
 * is O = 0, lse = -inf.
 *   o_parts [n_parts][n_rows][d], lse_parts [n_parts][n_rows]  (double)
 *   o [n_rows][d], lse [n_rows] or NULL                       (double)
 */
int oracle_merge_lse(int n_parts, int64_t n_rows, int d, const double* o_parts,
                     const double* lse_parts, double* o, double* lse) {
  if (n_parts < 1 || n_rows < 0 || d < 1 || !o_parts || !lse_parts || !o) return -1;
  for (int64_t r = 0; r < n_rows; ++r) {
    double mx = -INFINITY;
    for (int k = 0; k < n_parts; ++k)
      if (lse_parts[(int64_t)k * n_rows + r] > mx) mx = lse_parts[(int64_t)k * n_rows + r];
    for (int c = 0; c < d; ++c) o[r * d + c] = 0.0;
    if (mx == -INFINITY) {
      if (lse) lse[r] = -INFINITY;
      continue;
    }
    double total = 0.0;
    for (int k = 0; k < n_parts; ++k) {
      double l = lse_parts[(int64_t)k * n_rows + r];
      if (l == -INFINITY) continue;
      total += exp(l - mx);
    }
    double lse_r = mx + log(total);
    for (int k = 0; k < n_parts; ++k) {
      double l = lse_parts[(int64_t)k * n_rows + r];
      if (l == -INFINITY) continue;
      double w = exp(l - lse_r);
      for (int c = 0; c < d; ++c) o[r * d + c] += w * o_parts[((int64_t)k * n_rows + r) * d + c];
    }
    if (lse) lse[r] = lse_r;
  }
  return 0;
}

/*
 * SnapKV-style selection of the static draft cache at prefill (the static
 * selection the paper finds best, Sec. 4.4, Sec. 5.2; its footnote fixes an
 * observation window of 32 queries and average pooling with kernel 5).  The
 * steps restate the published SnapKV algorithm.
 *
 * oracle_snapkv_votes: for sequence b (prompt length S = kv_lens[b]) and kv
 * head hk, with the n_obs observation queries at positions
 * p_o = S - n_obs + o (o = 0 .. n_obs-1):
 *   a_{h,o}(j) = softmax over keys j' <= p_o of scale * q[b,o,h,:] . k[b,j',hk,:]
 *   vote(j)    = sum over the G query heads h of kv head hk and over o of a_{h,o}(j),
 *                for prefix positions j in [0, S - n_obs)
 *   pooled(j)  = (1/pool) * sum_{t = j - pool/2}^{j + pool/2} vote(t), with vote = 0
 *                outside [0, S - n_obs) (zero padding counted in the divisor)
 *   q_obs  [B, n_obs, Hq, d];  k as in oracle_attention
 *   pooled [B][Hkv][stride] doubles; entries at j >= S - n_obs are set to 0
 */
int oracle_snapkv_votes(int B, int n_obs, int Hq, int Hkv, int d, int dtype, double scale,
                        const void* q_obs, const void* k, int64_t s_blk, int64_t s_tok,
                        int64_t s_head, int page_size, const int32_t* page_table, int max_pages,
                        const int32_t* kv_lens, int pool, int stride, double* pooled) {
  if (B < 0 || n_obs < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || d < 1 || pool < 1 || pool % 2 == 0)
    return -1;
  if (dtype != ORACLE_F32 && dtype != ORACLE_BF16) return -1;
  if (B == 0) return 0;
  if (!q_obs || !k || !kv_lens || !pooled || stride < 1) return -1;
  job_t a = {ORACLE_VERIFY, B, n_obs, Hq, Hkv, d, dtype, scale, q_obs, k, NULL, s_blk, s_tok,
             s_head, page_size, page_table, max_pages, kv_lens, 0, 1, NULL, NULL, NULL, 0,
             NULL, NULL, 0, 1, 0, 0};
  const int G = Hq / Hkv;
  for (int b = 0; b < B; ++b) {
    const int S = kv_lens[b];
    const int n = S - n_obs;
    if (n > stride) return -1;
    double* vote = (double*)calloc((size_t)(n > 0 ? n : 1), sizeof(double));
    double* score = (double*)malloc(sizeof(double) * (size_t)(S > 0 ? S : 1));
    if (!vote || !score) {
      free(vote);
      free(score);
      return -1;
    }
    for (int hk = 0; hk < Hkv; ++hk) {
      for (int j = 0; j < (n > 0 ? n : 1); ++j) vote[j] = 0.0;
      for (int g = 0; g < G; ++g) {
        const int h = hk * G + g;
        for (int o = 0; o < n_obs; ++o) {
          const int p = S - n_obs + o;
          const int64_t q_off = (((int64_t)b * n_obs + o) * Hq + h) * d;
          double m = -INFINITY;
          for (int j = 0; j <= p && j < S; ++j) {
            const int64_t k_off = kv_offset(&a, b, j, hk);
            double dot = 0.0;
            for (int c = 0; c < d; ++c)
              dot += load_elem(q_obs, dtype, q_off + c) * load_elem(k, dtype, k_off + c);
            score[j] = scale * dot;
            if (score[j] > m) m = score[j];
          }
          double Z = 0.0;
          for (int j = 0; j <= p && j < S; ++j) Z += exp(score[j] - m);
          for (int j = 0; j < n; ++j) vote[j] += exp(score[j] - m) / Z;
        }
      }
      double* out = pooled + ((int64_t)b * Hkv + hk) * stride;
      for (int j = 0; j < stride; ++j) out[j] = 0.0;
      for (int j = 0; j < n; ++j) {
        double s = 0.0;
        for (int t = j - pool / 2; t <= j + pool / 2; ++t)
          if (t >= 0 && t < n) s += vote[t];
        out[j] = s / pool;
      }
    }
    free(vote);
    free(score);
  }
  return 0;
}

/* qsort order for selection: larger value first, then smaller position. */
static const double* g_sel_vals;
static int sel_cmp(const void* x, const void* y) {
  const int i = *(const int*)x, j = *(const int*)y;
  if (g_sel_vals[i] > g_sel_vals[j]) return -1;
  if (g_sel_vals[i] < g_sel_vals[j]) return 1;
  return i < j ? -1 : (i > j);
}
static int asc_cmp(const void* x, const void* y) {
  const int i = *(const int*)x, j = *(const int*)y;
  return i < j ? -1 : (i > j);
}

/*
 * oracle_snapkv_select: per row r (a (sequence, kv head) pair) with
 * n = lens[r] - n_obs prefix positions, keep the `budget - n_obs` prefix
 * positions of largest value (ties: the smaller position), all of them if
 * there are fewer, then the n_obs observation positions [n, lens[r]);
 * write them ascending to idx[r][0 .. count) and count to counts[r].
 *   vals [rows][stride] double, idx [rows][budget] int32, counts [rows] int32
 * Not thread-safe (qsort comparator state).
 */
int oracle_snapkv_select(int rows, const double* vals, int stride, const int32_t* lens, int n_obs,
                         int budget, int32_t* idx, int32_t* counts) {
  if (rows < 0 || stride < 1 || n_obs < 0 || budget < n_obs || !vals || !lens || !idx || !counts)
    return -1;
  int* order = (int*)malloc(sizeof(int) * (size_t)stride);
  if (!order) return -1;
  for (int r = 0; r < rows; ++r) {
    const int S = lens[r];
    const int n = S - n_obs > 0 ? S - n_obs : 0;
    if (n > stride) {
      free(order);
      return -1;
    }
    for (int j = 0; j < n; ++j) order[j] = j;
    g_sel_vals = vals + (int64_t)r * stride;
    qsort(order, (size_t)n, sizeof(int), sel_cmp);
    int keep = budget - n_obs < n ? budget - n_obs : n;
    qsort(order, (size_t)keep, sizeof(int), asc_cmp);
    int32_t* out = idx + (int64_t)r * budget;
    int c = 0;
    for (int t = 0; t < keep; ++t) out[c++] = order[t];
    for (int j = n; j < S; ++j) out[c++] = j;
    counts[r] = c;
  }
  free(order);
  return 0;
}
