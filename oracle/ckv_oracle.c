/*
 * ckv_oracle.c -- plain, slow, fp64 CPU oracle (TEST INFRASTRUCTURE ONLY).
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may
 * load this library.  It shares no code with the HIP path.  Every function
 * below names the passage of the paper it follows; no blocking, fusion or
 * reordering is done beyond what the definition states.
 */
#include "ckv_oracle.h"

#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>

/* bf16 is the upper half of an IEEE-754 binary32; widening is exact. */
double ckvref_bf16_to_f64(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* Sec. 2.2, Sec. 4.1: the retrieval score of a position is the query's inner
 * product with that position's landmark; the landmark of a position is its
 * own key here.  A KV head is shared by the G query heads of its group and
 * carries a single index set, so a position's score is the largest scaled
 * logit among those G heads. */
void ckvref_unit_scores(int G, int d, int n, const uint16_t* q,
                        const uint16_t* keys, int64_t key_row_stride,
                        float scale, double* S) {
  const double sc = (double)scale;
  for (int j = 0; j < n; ++j) {
    const uint16_t* kr = keys + (int64_t)j * key_row_stride;
    double best = -INFINITY;
    for (int g = 0; g < G; ++g) {
      double dot = 0.0;
      for (int c = 0; c < d; ++c)
        dot += ckvref_bf16_to_f64(q[g * d + c]) * ckvref_bf16_to_f64(kr[c]);
      double s = sc * dot;
      if (s > best) best = s;
    }
    S[j] = best;
  }
}

static _Thread_local const double* g_sort_scores;

/* Order of the critical set: larger score first; equal scores keep the lower
 * position first. */
static int by_score_desc(const void* a, const void* b) {
  int32_t i = *(const int32_t*)a, j = *(const int32_t*)b;
  double si = g_sort_scores[i], sj = g_sort_scores[j];
  if (si > sj) return -1;
  if (si < sj) return 1;
  return (i > j) - (i < j);
}

static int by_position(const void* a, const void* b) {
  int32_t i = *(const int32_t*)a, j = *(const int32_t*)b;
  return (i > j) - (i < j);
}

/* Sec. 2.2: only the important entries are retrieved, within the sparse
 * budget k.  Full sort of all positions by the order above, keep the first
 * m = min(k, n), then list them by ascending position. */
int ckvref_unit_select(int n, const double* S, int k, int32_t* idx) {
  int m = n < k ? n : k;
  if (m < 0) m = 0;
  if (n > 0) {
    int32_t* order = (int32_t*)malloc(sizeof(int32_t) * (size_t)n);
    for (int j = 0; j < n; ++j) order[j] = j;
    g_sort_scores = S;
    qsort(order, (size_t)n, sizeof(int32_t), by_score_desc);
    qsort(order, (size_t)m, sizeof(int32_t), by_position);
    memcpy(idx, order, sizeof(int32_t) * (size_t)m);
    free(order);
  }
  for (int i = m; i < k; ++i) idx[i] = -1;
  return m;
}

/* Sec. 5.3 / Sec. 5.4: the attention of the decoding token runs over exactly
 * the assembled sparse set.  Naive max-shifted softmax over the m logits,
 * then the probability-weighted sum of the value rows. */
void ckvref_unit_attn(int G, int d, int m, const uint16_t* q,
                      const uint16_t* k_rows, const uint16_t* v_rows,
                      float scale, double* out, double* p) {
  const double sc = (double)scale;
  double* logit = (double*)malloc(sizeof(double) * (size_t)(m > 0 ? m : 1));
  for (int g = 0; g < G; ++g) {
    double* o = out + (int64_t)g * d;
    for (int c = 0; c < d; ++c) o[c] = 0.0;
    if (m == 0) continue;
    double mx = -INFINITY;
    for (int i = 0; i < m; ++i) {
      double dot = 0.0;
      for (int c = 0; c < d; ++c)
        dot += ckvref_bf16_to_f64(q[g * d + c]) *
               ckvref_bf16_to_f64(k_rows[(int64_t)i * d + c]);
      logit[i] = sc * dot;
      if (logit[i] > mx) mx = logit[i];
    }
    double z = 0.0;
    for (int i = 0; i < m; ++i) {
      logit[i] = exp(logit[i] - mx);
      z += logit[i];
    }
    for (int i = 0; i < m; ++i) {
      double w = logit[i] / z;
      if (p) p[(int64_t)g * m + i] = w;
      for (int c = 0; c < d; ++c)
        o[c] += w * ckvref_bf16_to_f64(v_rows[(int64_t)i * d + c]);
    }
  }
  free(logit);
}

/* ------------------------------------------------------------------------ */
/* whole-batch wrappers                                                      */

static int shape_ok(const ckvref_shape* s) {
  if (!s) return 0;
  if (s->batch < 0 || s->num_q_heads < 1 || s->num_kv_heads < 1) return 0;
  if (s->num_q_heads % s->num_kv_heads) return 0;
  if (s->head_dim < 1 || s->max_ctx < 0) return 0;
  if (s->key_row_stride < s->head_dim || s->kv_row_stride < s->head_dim)
    return 0;
  return 1;
}

static int clamp_len(int32_t n, int32_t max_ctx) {
  if (n < 0) return 0;
  return n > max_ctx ? max_ctx : n;
}

typedef struct {
  const ckvref_shape* s;
  int kind; /* 0 score, 1 select, 2 attn, 3 pipeline, 4 dual-token attn */
  const uint16_t *q, *q2, *keys, *k_src, *v_src, *k_buf, *v_buf, *k_local, *v_local;
  double* out2;
  const int32_t* ctx_lens;
  const int32_t* n_sel_in;
  const double* scores_in;
  double* scores;
  int32_t* idx;
  int32_t* n_sel;
  double* out;
  int k;
  float scale;
  int unit_begin, unit_end;
} job;

static void run_unit(const job* jb, int u) {
  const ckvref_shape* s = jb->s;
  const int Hkv = s->num_kv_heads, G = s->num_q_heads / s->num_kv_heads;
  const int d = s->head_dim, nmax = s->max_ctx, k = jb->k;
  const int b = u / Hkv, h = u % Hkv;
  const int64_t qoff = ((int64_t)b * s->num_q_heads + (int64_t)h * G) * d;
  if (jb->kind == 0) {
    int n = clamp_len(jb->ctx_lens[b], nmax);
    double* S = jb->scores + (int64_t)u * nmax;
    ckvref_unit_scores(G, d, n, jb->q + qoff,
                       jb->keys + (int64_t)u * nmax * s->key_row_stride,
                       s->key_row_stride, jb->scale, S);
    for (int j = n; j < nmax; ++j) S[j] = -INFINITY;
  } else if (jb->kind == 1) {
    int n = clamp_len(jb->ctx_lens[b], nmax);
    jb->n_sel[u] = ckvref_unit_select(n, jb->scores_in + (int64_t)u * nmax, k,
                                      jb->idx + (int64_t)u * k);
  } else if (jb->kind == 2) {
    int m = jb->n_sel_in[u];
    if (m < 0) m = 0;
    if (m > k) m = k;
    ckvref_unit_attn(G, d, m, jb->q + qoff,
                     jb->k_buf + (int64_t)u * k * d,
                     jb->v_buf + (int64_t)u * k * d, jb->scale,
                     jb->out + qoff, NULL);
  } else if (jb->kind == 4) {
    /* Sec. 5.2: the two tokens as consecutive positions after the selected
     * rows; the causal mask hides the speculative token from the current
     * one.  Rows: the m buffer rows, then the local rows each token sees. */
    int m = jb->n_sel_in[u];
    if (m < 0) m = 0;
    if (m > k) m = k;
    uint16_t* kr = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)(m + 2) * d);
    uint16_t* vr = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)(m + 2) * d);
    memcpy(kr, jb->k_buf + (int64_t)u * k * d, sizeof(uint16_t) * (size_t)m * d);
    memcpy(vr, jb->v_buf + (int64_t)u * k * d, sizeof(uint16_t) * (size_t)m * d);
    memcpy(kr + (int64_t)m * d, jb->k_local + (int64_t)u * 2 * d, sizeof(uint16_t) * 2 * d);
    memcpy(vr + (int64_t)m * d, jb->v_local + (int64_t)u * 2 * d, sizeof(uint16_t) * 2 * d);
    ckvref_unit_attn(G, d, m + 1, jb->q + qoff, kr, vr, jb->scale, jb->out + qoff, NULL);
    ckvref_unit_attn(G, d, m + 2, jb->q2 + qoff, kr, vr, jb->scale, jb->out2 + qoff, NULL);
    free(kr);
    free(vr);
  } else {
    /* Sec. 4.1 + Sec. 5.3: index from the selecting query, attention of
     * the attending query over the rows of that index. */
    int n = clamp_len(jb->ctx_lens[b], nmax);
    double* S = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    ckvref_unit_scores(G, d, n, jb->q2 + qoff,
                       jb->keys + (int64_t)u * nmax * s->key_row_stride,
                       s->key_row_stride, jb->scale, S);
    int32_t* idx = jb->idx + (int64_t)u * k;
    int m = ckvref_unit_select(n, S, k, idx);
    jb->n_sel[u] = m;
    uint16_t* kr = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)(m > 0 ? m : 1) * d);
    uint16_t* vr = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)(m > 0 ? m : 1) * d);
    const int64_t base = (int64_t)u * nmax * s->kv_row_stride;
    for (int i = 0; i < m; ++i) {
      memcpy(kr + (int64_t)i * d,
             jb->k_src + base + (int64_t)idx[i] * s->kv_row_stride,
             sizeof(uint16_t) * d);
      memcpy(vr + (int64_t)i * d,
             jb->v_src + base + (int64_t)idx[i] * s->kv_row_stride,
             sizeof(uint16_t) * d);
    }
    ckvref_unit_attn(G, d, m, jb->q + qoff, kr, vr, jb->scale, jb->out + qoff,
                     NULL);
    free(kr);
    free(vr);
    free(S);
  }
}

static void* run_range(void* arg) {
  const job* jb = (const job*)arg;
  for (int u = jb->unit_begin; u < jb->unit_end; ++u) run_unit(jb, u);
  return NULL;
}

/* Units are independent; threads only split the unit range. */
static void run_units(job* base, int units, int nthreads) {
  if (nthreads < 1) nthreads = 1;
  if (nthreads > units) nthreads = units > 0 ? units : 1;
  if (nthreads == 1) {
    base->unit_begin = 0;
    base->unit_end = units;
    run_range(base);
    return;
  }
  pthread_t* th = (pthread_t*)malloc(sizeof(pthread_t) * (size_t)nthreads);
  job* jobs = (job*)malloc(sizeof(job) * (size_t)nthreads);
  for (int t = 0; t < nthreads; ++t) {
    jobs[t] = *base;
    jobs[t].unit_begin = (int)((int64_t)units * t / nthreads);
    jobs[t].unit_end = (int)((int64_t)units * (t + 1) / nthreads);
    pthread_create(&th[t], NULL, run_range, &jobs[t]);
  }
  for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
  free(jobs);
  free(th);
}

int ckvref_score_keys(const ckvref_shape* s, const uint16_t* q,
                      const uint16_t* k_score, const int32_t* ctx_lens,
                      float scale, double* scores, int nthreads) {
  if (!shape_ok(s)) return -1;
  job jb;
  memset(&jb, 0, sizeof jb);
  jb.s = s;
  jb.kind = 0;
  jb.q = q;
  jb.keys = k_score;
  jb.ctx_lens = ctx_lens;
  jb.scale = scale;
  jb.scores = scores;
  run_units(&jb, s->batch * s->num_kv_heads, nthreads);
  return 0;
}

int ckvref_select_topk(const ckvref_shape* s, const double* scores,
                       const int32_t* ctx_lens, int k, int32_t* idx,
                       int32_t* n_sel, int nthreads) {
  if (!shape_ok(s) || k < 1) return -1;
  job jb;
  memset(&jb, 0, sizeof jb);
  jb.s = s;
  jb.kind = 1;
  jb.scores_in = scores;
  jb.ctx_lens = ctx_lens;
  jb.k = k;
  jb.idx = idx;
  jb.n_sel = n_sel;
  run_units(&jb, s->batch * s->num_kv_heads, nthreads);
  return 0;
}

/* Sec. 5.4 (sparse KV assembly): each selected entry is placed, unchanged,
 * at its slot of the attention layout.  Slots i >= n_sel are not written. */
int ckvref_gather_kv(const ckvref_shape* s, const uint16_t* k_src,
                     const uint16_t* v_src, const int32_t* idx,
                     const int32_t* n_sel, int k, uint16_t* k_dst,
                     uint16_t* v_dst) {
  if (!shape_ok(s) || k < 1) return -1;
  const int units = s->batch * s->num_kv_heads, d = s->head_dim;
  for (int u = 0; u < units; ++u) {
    int m = n_sel[u];
    if (m > k) m = k;
    const int64_t base = (int64_t)u * s->max_ctx * s->kv_row_stride;
    for (int i = 0; i < m; ++i) {
      int64_t row = idx[(int64_t)u * k + i];
      memcpy(k_dst + ((int64_t)u * k + i) * d,
             k_src + base + row * s->kv_row_stride, sizeof(uint16_t) * d);
      memcpy(v_dst + ((int64_t)u * k + i) * d,
             v_src + base + row * s->kv_row_stride, sizeof(uint16_t) * d);
    }
  }
  return 0;
}

int ckvref_sparse_decode_attn(const ckvref_shape* s, const uint16_t* q_att,
                              const uint16_t* k_buf, const uint16_t* v_buf,
                              const int32_t* n_sel, int k, float scale,
                              double* out, int nthreads) {
  if (!shape_ok(s) || k < 1) return -1;
  job jb;
  memset(&jb, 0, sizeof jb);
  jb.s = s;
  jb.kind = 2;
  jb.q = q_att;
  jb.k_buf = k_buf;
  jb.v_buf = v_buf;
  jb.n_sel_in = n_sel;
  jb.k = k;
  jb.scale = scale;
  jb.out = out;
  run_units(&jb, s->batch * s->num_kv_heads, nthreads);
  return 0;
}

int ckvref_critical_kv_attn(const ckvref_shape* s, const uint16_t* q_att,
                            const uint16_t* q_sel, const uint16_t* k_score,
                            const uint16_t* k_src, const uint16_t* v_src,
                            const int32_t* ctx_lens, int k, float scale,
                            int32_t* idx, int32_t* n_sel, double* out,
                            int nthreads) {
  if (!shape_ok(s) || k < 1) return -1;
  job jb;
  memset(&jb, 0, sizeof jb);
  jb.s = s;
  jb.kind = 3;
  jb.q = q_att;
  jb.q2 = q_sel ? q_sel : q_att;
  jb.keys = k_score;
  jb.k_src = k_src;
  jb.v_src = v_src;
  jb.ctx_lens = ctx_lens;
  jb.k = k;
  jb.scale = scale;
  jb.idx = idx;
  jb.n_sel = n_sel;
  jb.out = out;
  run_units(&jb, s->batch * s->num_kv_heads, nthreads);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* chunk landmarks                                                           */

/* Round to 8 significant bits (bf16), ties to even: |x| = m * 2^e with m in
 * [0.5, 1) has quantum 2^(e-8); below the smallest normal bf16 (2^-126) the
 * quantum stays 2^-133.  nearbyint rounds ties to even in the default mode. */
uint16_t ckvref_f64_to_bf16(double x) {
  const uint16_t sign = signbit(x) ? 0x8000u : 0u;
  const double a = fabs(x);
  if (a == 0.0) return sign;
  int e;
  (void)frexp(a, &e);
  int q = e - 8;
  if (q < -133) q = -133;
  const double y = ldexp(nearbyint(ldexp(a, -q)), q);
  const float f = (float)y; /* exact: at most 8 significant bits */
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  return (uint16_t)(sign | (u >> 16));
}

/* Sec. 2.2: one landmark per chunk of adjacent entries, here their mean key;
 * Sec. 4.1: computed once, before decoding.  Only rows below n_b count. */
int ckvref_chunk_landmarks(const ckvref_shape* s, int chunk, const uint16_t* keys,
                           const int32_t* ctx_lens, uint16_t* landmarks) {
  if (!shape_ok(s) || chunk < 1) return -1;
  const int units = s->batch * s->num_kv_heads, d = s->head_dim;
  const int nmax = s->max_ctx, cmax = (nmax + chunk - 1) / chunk;
  for (int u = 0; u < units; ++u) {
    const int n = clamp_len(ctx_lens[u / s->num_kv_heads], nmax);
    const int nc = (n + chunk - 1) / chunk;
    const uint16_t* ku = keys + (int64_t)u * nmax * s->key_row_stride;
    for (int c = 0; c < nc; ++c) {
      const int j0 = c * chunk, j1 = j0 + chunk < n ? j0 + chunk : n;
      for (int ch = 0; ch < d; ++ch) {
        double sum = 0.0;
        for (int j = j0; j < j1; ++j)
          sum += ckvref_bf16_to_f64(ku[(int64_t)j * s->key_row_stride + ch]);
        landmarks[((int64_t)u * cmax + c) * d + ch] = ckvref_f64_to_bf16(sum / (j1 - j0));
      }
    }
  }
  return 0;
}

/* Sec. 2.2: a selected chunk brings all of its (valid) entries. */
int ckvref_expand_chunks(int chunk, int m, const int32_t* chunk_idx, int n, int k,
                         int32_t* rows) {
  int r = 0;
  for (int i = 0; i < m; ++i)
    for (int t = 0; t < chunk; ++t) {
      const int row = chunk_idx[i] * chunk + t;
      if (row < n && r < k) rows[r++] = row;
    }
  for (int i = r; i < k; ++i) rows[i] = -1;
  return r;
}

int ckvref_select_chunks(const ckvref_shape* s, int chunk, const uint16_t* q_sel,
                         const uint16_t* landmarks, const int32_t* ctx_lens, int k,
                         float scale, int32_t* chunk_idx, int32_t* n_chunks,
                         int32_t* rows, int32_t* n_rows, int nthreads) {
  if (!shape_ok(s) || chunk < 1 || k < chunk || k % chunk) return -1;
  const int units = s->batch * s->num_kv_heads, kc = k / chunk;
  const int cmax = (s->max_ctx + chunk - 1) / chunk;
  /* the landmarks as a batch of rows: one per chunk, ceil(n_b/chunk) valid */
  ckvref_shape sc = *s;
  sc.max_ctx = cmax;
  sc.key_row_stride = s->head_dim;
  sc.kv_row_stride = s->head_dim;
  int32_t* clens = (int32_t*)malloc(sizeof(int32_t) * (size_t)(s->batch > 0 ? s->batch : 1));
  for (int b = 0; b < s->batch; ++b)
    clens[b] = (clamp_len(ctx_lens[b], s->max_ctx) + chunk - 1) / chunk;
  double* S = (double*)malloc(sizeof(double) * (size_t)units * (size_t)(cmax > 0 ? cmax : 1));
  ckvref_score_keys(&sc, q_sel, landmarks, clens, scale, S, nthreads);
  ckvref_select_topk(&sc, S, clens, kc, chunk_idx, n_chunks, nthreads);
  for (int u = 0; u < units; ++u) {
    const int n = clamp_len(ctx_lens[u / s->num_kv_heads], s->max_ctx);
    n_rows[u] = ckvref_expand_chunks(chunk, n_chunks[u], chunk_idx + (int64_t)u * kc, n, k,
                                     rows + (int64_t)u * k);
  }
  free(S);
  free(clens);
  return 0;
}

int ckvref_dual_token_attn(const ckvref_shape* s, const uint16_t* q_cur,
                           const uint16_t* q_spec, const uint16_t* k_buf,
                           const uint16_t* v_buf, const int32_t* n_sel,
                           const uint16_t* k_local, const uint16_t* v_local, int k,
                           float scale, double* out_cur, double* out_spec, int nthreads) {
  if (!shape_ok(s) || k < 1) return -1;
  job jb;
  memset(&jb, 0, sizeof jb);
  jb.s = s;
  jb.kind = 4;
  jb.q = q_cur;
  jb.q2 = q_spec;
  jb.k_buf = k_buf;
  jb.v_buf = v_buf;
  jb.n_sel_in = n_sel;
  jb.k_local = k_local;
  jb.v_local = v_local;
  jb.k = k;
  jb.scale = scale;
  jb.out = out_cur;
  jb.out2 = out_spec;
  run_units(&jb, s->batch * s->num_kv_heads, nthreads);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* low-rank key reconstruction                                               */

/* Sec. 5.3: a selected key is rebuilt from the unit's low-rank factors. */
int ckvref_reconstruct_keys(const ckvref_shape* s, int rank, const uint16_t* u_fac,
                            const uint16_t* w_fac, const int32_t* idx, const int32_t* n_sel,
                            int k, uint16_t* k_dst) {
  if (!shape_ok(s) || rank < 1 || k < 1) return -1;
  const int units = s->batch * s->num_kv_heads, d = s->head_dim;
  for (int u = 0; u < units; ++u) {
    int m = n_sel[u];
    if (m < 0) m = 0;
    if (m > k) m = k;
    const uint16_t* W = w_fac + (int64_t)u * rank * d;
    for (int i = 0; i < m; ++i) {
      const uint16_t* U = u_fac + ((int64_t)u * s->max_ctx + idx[(int64_t)u * k + i]) * rank;
      for (int c = 0; c < d; ++c) {
        double acc = 0.0;
        for (int j = 0; j < rank; ++j)
          acc += ckvref_bf16_to_f64(U[j]) * ckvref_bf16_to_f64(W[(int64_t)j * d + c]);
        k_dst[((int64_t)u * k + i) * d + c] = ckvref_f64_to_bf16(acc);
      }
    }
  }
  return 0;
}
