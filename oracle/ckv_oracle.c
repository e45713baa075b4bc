/*
 * ckv_oracle.c -- CPU oracle for the ContiguousKV Re-Prefill hot path.
 *
 * TEST INFRASTRUCTURE ONLY: the fp64 reference the GPU library is checked
 * against.  Loaded only by the tests, the smoke check and the benchmark's
 * CPU-baseline leg.  Shares no code with the GPU library.
 *
 * Build: gcc -std=c11 -O2 -ffp-contract=off -fno-fast-math -fPIC -shared -pthread
 * (no contraction of a*b+c into fma, no reassociation: every sum below is
 * evaluated in the order written).
 *
 * Arithmetic: every input element is widened exactly to double (bf16 bits are
 * the top half of an IEEE float), and all sums, exponentials and quotients are
 * fp64 in plain sequential loops.  Threads only split independent work: the
 * rows of the token-importance sum are cut into a fixed number of blocks whose
 * partial sums are added in block order, so no result depends on the thread
 * count.
 */
#define _GNU_SOURCE
#include "ckv_oracle.h"

#include <float.h>
#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

/* ------------------------------------------------------------------------- */
/* small helpers                                                              */
/* ------------------------------------------------------------------------- */

static double widen(const void* p, int dtype, int64_t i) {
  if (dtype == CKVO_F32) return (double)((const float*)p)[i];
  uint32_t bits = (uint32_t)((const uint16_t*)p)[i] << 16;
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

static double* widen_all(const void* p, int dtype, int64_t count) {
  double* out = (double*)malloc((size_t)(count > 0 ? count : 1) * sizeof(double));
  if (!out) return NULL;
  for (int64_t i = 0; i < count; ++i) out[i] = widen(p, dtype, i);
  return out;
}

static int elem_bytes(int dtype) { return dtype == CKVO_F32 ? 4 : 2; }

static int shape_ok(const ckvo_shape* s) {
  if (!s) return 0;
  if (s->n_prefix < 1 || s->n_suffix < 0 || s->n_q_heads < 1 || s->n_kv_heads < 1) return 0;
  if (s->n_q_heads % s->n_kv_heads != 0) return 0;
  if (s->head_dim < 1 || s->chunk_size < 1) return 0;
  if (s->dtype != CKVO_F32 && s->dtype != CKVO_BF16) return 0;
  if (!(s->sm_scale >= 0.0)) return 0;
  return 1;
}

static double scale_of(const ckvo_shape* s) {
  return s->sm_scale > 0.0 ? s->sm_scale : 1.0 / sqrt((double)s->head_dim);
}

static int resolve_threads(int nthreads) {
  if (nthreads > 0) return nthreads;
  long n = sysconf(_SC_NPROCESSORS_ONLN);
  return n > 0 ? (int)n : 1;
}

/* Runs fn(ctx, item) for item in [0, n_items) on nthreads threads.  Items are
 * claimed from a shared counter; each item must write only its own outputs. */
typedef void (*item_fn)(void* ctx, int64_t item, void* scratch);
typedef struct {
  item_fn fn;
  void* ctx;
  int64_t n_items;
  int64_t next;
  size_t scratch_bytes;
  int failed;
} pool_t;

static void* pool_worker(void* arg) {
  pool_t* p = (pool_t*)arg;
  void* scratch = malloc(p->scratch_bytes ? p->scratch_bytes : 1);
  if (!scratch) {
    __atomic_store_n(&p->failed, 1, __ATOMIC_SEQ_CST);
    return NULL;
  }
  for (;;) {
    int64_t it = __atomic_fetch_add(&p->next, 1, __ATOMIC_SEQ_CST);
    if (it >= p->n_items) break;
    p->fn(p->ctx, it, scratch);
  }
  free(scratch);
  return NULL;
}

static int run_pool(item_fn fn, void* ctx, int64_t n_items, size_t scratch_bytes, int nthreads) {
  pool_t p = {fn, ctx, n_items, 0, scratch_bytes, 0};
  int nt = resolve_threads(nthreads);
  if (nt > n_items) nt = (int)(n_items > 0 ? n_items : 1);
  pthread_t* th = (pthread_t*)malloc(sizeof(pthread_t) * (size_t)nt);
  if (!th) return -2;
  int started = 0;
  for (int i = 0; i < nt; ++i) {
    if (pthread_create(&th[i], NULL, pool_worker, &p) != 0) break;
    ++started;
  }
  if (started == 0) pool_worker(&p);
  for (int i = 0; i < started; ++i) pthread_join(th[i], NULL);
  free(th);
  return p.failed ? -2 : 0;
}

/* ------------------------------------------------------------------------- */
/* Def. 4.1 partition and the budget                                          */
/* ------------------------------------------------------------------------- */

int64_t ckvo_num_chunks(int64_t n, int32_t c) {
  if (n < 0 || c < 1) return -1;
  return (n + c - 1) / c;
}

int64_t ckvo_num_keep(int64_t m, double r) {
  if (!(r > 0.0 && r <= 1.0) || m < 0) return -1;
  if (m == 0) return 0;
  double x = ceil(r * (double)m - 1e-9);
  int64_t k = (int64_t)x;
  if (k < 1) k = 1;
  if (k > m) k = m;
  return k;
}

/* first token and length of chunk j (Def. 4.1; the last chunk may be short) */
static int64_t chunk_first(const ckvo_shape* s, int64_t j) { return j * s->chunk_size; }
static int64_t chunk_len(const ckvo_shape* s, int64_t j) {
  int64_t lo = j * s->chunk_size, hi = lo + s->chunk_size;
  if (hi > s->n_prefix) hi = s->n_prefix;
  return hi - lo;
}

/* ------------------------------------------------------------------------- */
/* Sec. 4.4 token importance                                                  */
/* ------------------------------------------------------------------------- */
/* Reading of the garbled passage: the probe matrix is (all suffix queries x all
 * query heads) by (prefix keys), the softmax runs over the prefix keys only, and
 * a token's importance is the sum of its column, i.e. the sum over the query
 * axis.  The logit is sm_scale * q.k (the paper's softmax omits the scale; the
 * standard 1/sqrt(d) is taken).  Rows are visited in (kv head g, head i of g's
 * group, query t) order. */

#define IMPORTANCE_BLOCKS 64

typedef struct {
  const ckvo_shape* s;
  const double* q;  /* [S][Hq][d] */
  const double* k;  /* [n][Hkv][d] */
  double* partial;  /* [blocks][n] */
  int64_t rows, blocks;
  double scale;
} imp_ctx;

static void importance_block(void* vctx, int64_t b, void* scratch) {
  imp_ctx* c = (imp_ctx*)vctx;
  double* logit = (double*)scratch;
  const ckvo_shape* s = c->s;
  const int64_t n = s->n_prefix, S = s->n_suffix, Hq = s->n_q_heads, Hkv = s->n_kv_heads;
  const int64_t d = s->head_dim, G = Hq / Hkv;
  int64_t r0 = b * c->rows / c->blocks, r1 = (b + 1) * c->rows / c->blocks;
  double* acc = c->partial + b * n;
  for (int64_t r = r0; r < r1; ++r) {
    int64_t g = r / (G * S), i = (r / S) % G, t = r % S;
    int64_t h = g * G + i;
    const double* qr = c->q + (t * Hq + h) * d;
    double mx = -INFINITY;
    for (int64_t x = 0; x < n; ++x) {
      const double* kx = c->k + (x * Hkv + g) * d;
      double dot = 0.0;
      for (int64_t e = 0; e < d; ++e) dot += qr[e] * kx[e];
      logit[x] = c->scale * dot;
      if (logit[x] > mx) mx = logit[x];
    }
    double z = 0.0;
    for (int64_t x = 0; x < n; ++x) {
      logit[x] = exp(logit[x] - mx);
      z += logit[x];
    }
    for (int64_t x = 0; x < n; ++x) acc[x] += logit[x] / z;
  }
}

int ckvo_token_importance(const ckvo_shape* s, const void* q, const void* k_prefix, double* a,
                          int nthreads) {
  if (!shape_ok(s) || !q || !k_prefix || !a) return -1;
  const int64_t n = s->n_prefix;
  const int64_t rows = (int64_t)s->n_suffix * s->n_q_heads;
  for (int64_t x = 0; x < n; ++x) a[x] = 0.0;
  if (rows == 0) return 0;
  int64_t blocks = rows < IMPORTANCE_BLOCKS ? rows : IMPORTANCE_BLOCKS;
  double* qd = widen_all(q, s->dtype, rows * s->head_dim);
  double* kd = widen_all(k_prefix, s->dtype, n * s->n_kv_heads * s->head_dim);
  double* partial = (double*)calloc((size_t)(blocks * n), sizeof(double));
  int rc = -2;
  if (qd && kd && partial) {
    imp_ctx c = {s, qd, kd, partial, rows, blocks, scale_of(s)};
    rc = run_pool(importance_block, &c, blocks, (size_t)n * sizeof(double), nthreads);
    if (rc == 0)
      for (int64_t b = 0; b < blocks; ++b)
        for (int64_t x = 0; x < n; ++x) a[x] += partial[b * n + x];
  }
  free(qd);
  free(kd);
  free(partial);
  return rc;
}

/* Eq. 1: A_j is the sum of a_i over chunk j's tokens (0-based j; the range in
 * the equation, c*j .. c*j+c-1, is taken over the prose's c*(j-1) .. c*j, which
 * would hold c+1 tokens; the last chunk is clamped to n). */
int ckvo_chunk_scores(const ckvo_shape* s, const double* a, double* A) {
  if (!shape_ok(s) || !a || !A) return -1;
  int64_t m = ckvo_num_chunks(s->n_prefix, s->chunk_size);
  for (int64_t j = 0; j < m; ++j) {
    double sum = 0.0;
    int64_t first = chunk_first(s, j), len = chunk_len(s, j);
    for (int64_t x = first; x < first + len; ++x) sum += a[x];
    A[j] = sum;
  }
  return 0;
}

/* ------------------------------------------------------------------------- */
/* top-k selection                                                            */
/* ------------------------------------------------------------------------- */
/* The paper ranks chunks by A_j and keeps the highest-scoring k.  It names no
 * tie-break; the lowest chunk index wins among equal scores.  The result is a
 * set, reported in ascending chunk order. */

static const double* g_sort_scores; /* only used under g_sort_lock */
static pthread_mutex_t g_sort_lock = PTHREAD_MUTEX_INITIALIZER;

static int rank_cmp(const void* pa, const void* pb) {
  int32_t ia = *(const int32_t*)pa, ib = *(const int32_t*)pb;
  double x = g_sort_scores[ia], y = g_sort_scores[ib];
  int xn = isnan(x), yn = isnan(y);
  if (xn != yn) return xn ? 1 : -1; /* NaN ranks last */
  if (!xn) {
    if (x > y) return -1; /* higher score first; -0.0 == +0.0 here */
    if (x < y) return 1;
  }
  return (ia > ib) - (ia < ib); /* then lower index first */
}

static int int_cmp(const void* pa, const void* pb) {
  int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
  return (a > b) - (a < b);
}

int ckvo_select_topk(const double* A, int64_t m, int64_t k, int32_t* sel) {
  if (!A || !sel || m < 1 || m > INT32_MAX || k < 1 || k > m) return -1;
  int32_t* order = (int32_t*)malloc(sizeof(int32_t) * (size_t)m);
  if (!order) return -2;
  for (int64_t j = 0; j < m; ++j) order[j] = (int32_t)j;
  pthread_mutex_lock(&g_sort_lock);
  g_sort_scores = A;
  qsort(order, (size_t)m, sizeof(int32_t), rank_cmp);
  g_sort_scores = NULL;
  pthread_mutex_unlock(&g_sort_lock);
  memcpy(sel, order, sizeof(int32_t) * (size_t)k);
  qsort(sel, (size_t)k, sizeof(int32_t), int_cmp);
  free(order);
  return 0;
}

/* ------------------------------------------------------------------------- */
/* Def. 2.1 re-prefill attention                                              */
/* ------------------------------------------------------------------------- */
/* Query t of head h attends to a key sequence; weights are the softmax of
 * sm_scale * q.k over that sequence (max subtracted), and the output is the
 * weighted sum of the matching values.  The suffix is attended causally (query
 * t sees suffix tokens 0..t) and is never pruned. */

typedef struct {
  const ckvo_shape* s;
  const double *q, *kp, *vp, *ks, *vs;
  const int32_t* sel; /* NULL: dense */
  int64_t k;
  const int64_t* row_ids;
  int64_t n_rows;
  double* out;
  double scale;
  int64_t max_keys; /* longest key sequence of any row */
} attn_ctx;

/* Builds the key sequence of query t in KV head g as row pointers into the
 * widened K and V tensors, in attention order; returns its length. */
static int64_t collect_keys(const attn_ctx* c, int64_t t, int64_t g, const double** krow,
                            const double** vrow) {
  const ckvo_shape* s = c->s;
  const int64_t Hkv = s->n_kv_heads, d = s->head_dim;
  int64_t nk = 0;
  if (c->sel) {
    for (int64_t u = 0; u < c->k; ++u) {
      int64_t first = chunk_first(s, c->sel[u]), len = chunk_len(s, c->sel[u]);
      for (int64_t x = first; x < first + len; ++x) {
        krow[nk] = c->kp + (x * Hkv + g) * d;
        vrow[nk] = c->vp + (x * Hkv + g) * d;
        ++nk;
      }
    }
  } else {
    for (int64_t x = 0; x < s->n_prefix; ++x) {
      krow[nk] = c->kp + (x * Hkv + g) * d;
      vrow[nk] = c->vp + (x * Hkv + g) * d;
      ++nk;
    }
  }
  for (int64_t x = 0; x <= t; ++x) {
    krow[nk] = c->ks + (x * Hkv + g) * d;
    vrow[nk] = c->vs + (x * Hkv + g) * d;
    ++nk;
  }
  return nk;
}

static void attn_row(void* vctx, int64_t r, void* scratch) {
  attn_ctx* c = (attn_ctx*)vctx;
  const ckvo_shape* s = c->s;
  const int64_t Hq = s->n_q_heads, Hkv = s->n_kv_heads, d = s->head_dim, G = Hq / Hkv;
  int64_t id = c->row_ids ? c->row_ids[r] : r;
  int64_t t = id / Hq, h = id % Hq, g = h / G;
  const double* qr = c->q + (t * Hq + h) * d;
  double* o = c->out + (c->row_ids ? r : id) * d;

  double* w = (double*)scratch;
  const double** krow = (const double**)(w + c->max_keys);
  const double** vrow = krow + c->max_keys;
  int64_t nk = collect_keys(c, t, g, krow, vrow);

  double mx = -INFINITY;
  for (int64_t x = 0; x < nk; ++x) {
    double dot = 0.0;
    for (int64_t e = 0; e < d; ++e) dot += qr[e] * krow[x][e];
    w[x] = c->scale * dot;
    if (w[x] > mx) mx = w[x];
  }
  double z = 0.0;
  for (int64_t x = 0; x < nk; ++x) {
    w[x] = exp(w[x] - mx);
    z += w[x];
  }
  for (int64_t e = 0; e < d; ++e) o[e] = 0.0;
  for (int64_t x = 0; x < nk; ++x) {
    double p = w[x] / z;
    for (int64_t e = 0; e < d; ++e) o[e] += p * vrow[x][e];
  }
}

static int attn_common(const ckvo_shape* s, const void* q, const void* k_prefix,
                       const void* v_prefix, const int32_t* sel, int64_t k, const void* k_suffix,
                       const void* v_suffix, const int64_t* row_ids, int64_t n_rows, double* out,
                       int nthreads) {
  const int64_t S = s->n_suffix, Hq = s->n_q_heads, Hkv = s->n_kv_heads, d = s->head_dim;
  const int64_t n = s->n_prefix;
  int64_t total = row_ids ? n_rows : S * Hq;
  if (row_ids)
    for (int64_t r = 0; r < n_rows; ++r)
      if (row_ids[r] < 0 || row_ids[r] >= S * Hq) return -1;
  if (total == 0) return 0;
  double* qd = widen_all(q, s->dtype, S * Hq * d);
  double* kp = widen_all(k_prefix, s->dtype, n * Hkv * d);
  double* vp = widen_all(v_prefix, s->dtype, n * Hkv * d);
  double* ks = widen_all(k_suffix, s->dtype, S * Hkv * d);
  double* vs = widen_all(v_suffix, s->dtype, S * Hkv * d);
  int rc = -2;
  if (qd && kp && vp && ks && vs) {
    int64_t max_keys = (sel ? k * s->chunk_size : n) + S;
    attn_ctx c = {s, qd, kp, vp, ks, vs, sel, k, row_ids, n_rows, out, scale_of(s), max_keys};
    rc = run_pool(attn_row, &c, total, (size_t)max_keys * 3 * sizeof(double), nthreads);
  }
  free(qd);
  free(kp);
  free(vp);
  free(ks);
  free(vs);
  return rc;
}

int ckvo_sparse_attn(const ckvo_shape* s, const void* q, const void* k_prefix,
                     const void* v_prefix, const int32_t* sel, int64_t k, const void* k_suffix,
                     const void* v_suffix, const int64_t* row_ids, int64_t n_rows, double* out,
                     int nthreads) {
  if (!shape_ok(s) || !q || !k_prefix || !v_prefix || !sel || !out) return -1;
  if (s->n_suffix > 0 && (!k_suffix || !v_suffix)) return -1;
  int64_t m = ckvo_num_chunks(s->n_prefix, s->chunk_size);
  if (k < 0 || k > m) return -1;
  for (int64_t u = 0; u < k; ++u) {
    if (sel[u] < 0 || sel[u] >= m) return -1;
    if (u > 0 && sel[u] <= sel[u - 1]) return -1;
  }
  return attn_common(s, q, k_prefix, v_prefix, sel, k, k_suffix, v_suffix, row_ids, n_rows, out,
                     nthreads);
}

int ckvo_dense_attn(const ckvo_shape* s, const void* q, const void* k_prefix,
                    const void* v_prefix, const void* k_suffix, const void* v_suffix,
                    const int64_t* row_ids, int64_t n_rows, double* out, int nthreads) {
  if (!shape_ok(s) || !q || !k_prefix || !v_prefix || !out) return -1;
  if (s->n_suffix > 0 && (!k_suffix || !v_suffix)) return -1;
  return attn_common(s, q, k_prefix, v_prefix, NULL, 0, k_suffix, v_suffix, row_ids, n_rows, out,
                     nthreads);
}

/* ------------------------------------------------------------------------- */
/* Sec. 4.2 contiguous gather and Sec. 4.3.2 prefetch accounting              */
/* ------------------------------------------------------------------------- */

int ckvo_gather_chunks(const ckvo_shape* s, const void* k_src, const void* v_src,
                       const int32_t* sel, int64_t k, void* k_dst, void* v_dst) {
  if (!shape_ok(s) || !k_src || !v_src || !sel || !k_dst || !v_dst) return -1;
  int64_t m = ckvo_num_chunks(s->n_prefix, s->chunk_size);
  if (k < 0 || k > m) return -1;
  for (int64_t u = 0; u < k; ++u)
    if (sel[u] < 0 || sel[u] >= m) return -1;
  const size_t row = (size_t)s->n_kv_heads * (size_t)s->head_dim * (size_t)elem_bytes(s->dtype);
  const size_t slot = row * (size_t)s->chunk_size;
  for (int64_t u = 0; u < k; ++u) {
    size_t src = (size_t)chunk_first(s, sel[u]) * row;
    size_t len = (size_t)chunk_len(s, sel[u]) * row;
    memcpy((char*)k_dst + u * slot, (const char*)k_src + src, len);
    memcpy((char*)v_dst + u * slot, (const char*)v_src + src, len);
    memset((char*)k_dst + u * slot + len, 0, slot - len);
    memset((char*)v_dst + u * slot + len, 0, slot - len);
  }
  return 0;
}

int ckvo_layer_accounting(const ckvo_shape* s, const int32_t* sel, int64_t k,
                          const int32_t* pred, int64_t n_pred, ckvo_layer_stats* st) {
  if (!shape_ok(s) || !st || k < 0 || n_pred < 0) return -1;
  if ((k > 0 && !sel) || (n_pred > 0 && !pred)) return -1;
  int64_t m = ckvo_num_chunks(s->n_prefix, s->chunk_size);
  for (int64_t u = 0; u < k; ++u)
    if (sel[u] < 0 || sel[u] >= m || (u > 0 && sel[u] <= sel[u - 1])) return -1;
  for (int64_t u = 0; u < n_pred; ++u)
    if (pred[u] < 0 || pred[u] >= m || (u > 0 && pred[u] <= pred[u - 1])) return -1;
  const int64_t per_token = 2LL * s->n_kv_heads * s->head_dim * elem_bytes(s->dtype);
  memset(st, 0, sizeof *st);
  st->k = k;
  int64_t a = 0, b = 0;
  while (a < k || b < n_pred) {
    if (b >= n_pred || (a < k && sel[a] < pred[b])) { /* needed, not prefetched */
      st->misses++;
      st->bytes_demand += chunk_len(s, sel[a]) * per_token;
      st->bytes_used += chunk_len(s, sel[a]) * per_token;
      ++a;
    } else if (a >= k || pred[b] < sel[a]) { /* prefetched, not needed */
      st->wasted++;
      st->bytes_prefetch += chunk_len(s, pred[b]) * per_token;
      ++b;
    } else { /* prefetched and needed */
      st->hits++;
      st->bytes_prefetch += chunk_len(s, pred[b]) * per_token;
      st->bytes_used += chunk_len(s, sel[a]) * per_token;
      ++a;
      ++b;
    }
  }
  return 0;
}

/* ------------------------------------------------------------------------- */
/* one layer                                                                  */
/* ------------------------------------------------------------------------- */

int ckvo_reprefill_layer(const ckvo_shape* s, double keep_ratio, const void* q,
                         const void* k_prefix, const void* v_prefix, const void* k_suffix,
                         const void* v_suffix, double* A, int32_t* sel, int64_t* k_out,
                         double* out, int nthreads) {
  if (!shape_ok(s) || !A || !sel || !k_out || !out) return -1;
  int64_t m = ckvo_num_chunks(s->n_prefix, s->chunk_size);
  int64_t k = ckvo_num_keep(m, keep_ratio);
  if (k < 1) return -1;
  double* a = (double*)malloc(sizeof(double) * (size_t)s->n_prefix);
  if (!a) return -2;
  int rc = ckvo_token_importance(s, q, k_prefix, a, nthreads);
  if (rc == 0) rc = ckvo_chunk_scores(s, a, A);
  if (rc == 0) rc = ckvo_select_topk(A, m, k, sel);
  if (rc == 0)
    rc = ckvo_sparse_attn(s, q, k_prefix, v_prefix, sel, k, k_suffix, v_suffix, NULL, 0, out,
                          nthreads);
  free(a);
  *k_out = k;
  return rc;
}

/* ------------------------------------------------------------------------- */
/* read accounting against a store of fixed blocks                           */
/* ------------------------------------------------------------------------- */

/* Sec. 4.2 and Sec. 3 (Motivation 1): mark every token of every selected
 * chunk, then visit the store's blocks of b consecutive tokens one by one; a
 * block with a marked token is read whole (the last block holds n mod b tokens
 * when b does not divide n). */
int ckvo_io_account(int64_t n, int32_t c, const int32_t* sel, int64_t k, int32_t b,
                    ckvo_io_counts* out) {
  if (n < 1 || c < 1 || b < 1 || k < 0 || !out || (k > 0 && !sel)) return -1;
  int64_t m = ckvo_num_chunks(n, c);
  if (k > m) return -1;
  unsigned char* chunk_marked = (unsigned char*)calloc((size_t)m, 1);
  unsigned char* token_marked = (unsigned char*)calloc((size_t)n, 1);
  if (!chunk_marked || !token_marked) {
    free(chunk_marked);
    free(token_marked);
    return -2;
  }
  int rc = 0;
  for (int64_t u = 0; u < k && rc == 0; ++u) {
    int64_t j = sel[u];
    if (j < 0 || j >= m || chunk_marked[j]) {
      rc = -1;
      break;
    }
    chunk_marked[j] = 1;
    for (int64_t t = j * c; t < (j + 1) * c && t < n; ++t) token_marked[t] = 1;
  }
  if (rc == 0) {
    memset(out, 0, sizeof *out);
    for (int64_t t = 0; t < n; ++t) out->tokens_selected += token_marked[t];
    for (int64_t j = 0; j < m; ++j)
      if (chunk_marked[j] && (j == 0 || !chunk_marked[j - 1])) out->runs++;
    for (int64_t first = 0; first < n; first += b) {
      int64_t last = first + b < n ? first + b : n;
      int any = 0;
      for (int64_t t = first; t < last; ++t) any |= token_marked[t];
      if (any) {
        out->blocks++;
        out->tokens_block += last - first;
      }
    }
  }
  free(chunk_marked);
  free(token_marked);
  return rc;
}

/* ------------------------------------------------------------------------- */
/* attention-guided cache                                                     */
/* ------------------------------------------------------------------------- */

struct ckvo_cache {
  int64_t n_keys, gpu_slots, cpu_slots;
  int policy;
  double* I;      /* cumulative importance: sum of A over the key's accesses */
  int64_t* F;     /* accesses (CKVO_CACHE_LOADS: loads into GPU or CPU memory) */
  int64_t* last;  /* time of the key's latest access (0: never) */
  int8_t* tier;
  int64_t clock;
  ckvo_cache_counts counts;
};

ckvo_cache* ckvo_cache_create(int64_t n_keys, int64_t gpu_slots, int64_t cpu_slots, int policy) {
  if (n_keys < 1 || gpu_slots < 0 || cpu_slots < 0) return NULL;
  if (policy != CKVO_CACHE_ATTENTION && policy != CKVO_CACHE_LFU && policy != CKVO_CACHE_LOADS)
    return NULL;
  ckvo_cache* c = (ckvo_cache*)calloc(1, sizeof *c);
  if (!c) return NULL;
  c->n_keys = n_keys;
  c->gpu_slots = gpu_slots;
  c->cpu_slots = cpu_slots;
  c->policy = policy;
  c->I = (double*)calloc((size_t)n_keys, sizeof(double));
  c->F = (int64_t*)calloc((size_t)n_keys, sizeof(int64_t));
  c->last = (int64_t*)calloc((size_t)n_keys, sizeof(int64_t));
  c->tier = (int8_t*)calloc((size_t)n_keys, 1);
  if (!c->I || !c->F || !c->last || !c->tier) {
    ckvo_cache_destroy(c);
    return NULL;
  }
  return c;
}

void ckvo_cache_destroy(ckvo_cache* c) {
  if (!c) return;
  free(c->I);
  free(c->F);
  free(c->last);
  free(c->tier);
  free(c);
}

/* Eq. 2: S = I * F; the frequency-only foil ranks by F alone. */
static double cache_score(const ckvo_cache* c, int64_t x) {
  if (c->policy == CKVO_CACHE_LFU) return (double)c->F[x];
  return c->I[x] * (double)c->F[x];
}

/* Eviction order: the lower score leaves first; among equal scores, the key
 * whose latest access is older. */
static int leaves_before(const ckvo_cache* c, int64_t x, int64_t y) {
  double sx = cache_score(c, x), sy = cache_score(c, y);
  if (sx != sy) return sx < sy;
  return c->last[x] < c->last[y];
}

/* The key of `tier` that leaves first (-1 if the tier is empty); *count gets
 * the tier's occupancy.  A linear scan over every key. */
static int64_t tier_first_out(const ckvo_cache* c, int tier, int64_t* count) {
  int64_t best = -1, cnt = 0;
  for (int64_t x = 0; x < c->n_keys; ++x) {
    if (c->tier[x] != tier) continue;
    ++cnt;
    if (best < 0 || leaves_before(c, x, best)) best = x;
  }
  *count = cnt;
  return best;
}

/* Places x in the CPU tier if there is room or x outranks the CPU tier's
 * weakest entry (which then leaves memory); otherwise x leaves memory.
 * Returns 1 when x was placed. */
static int admit_cpu(ckvo_cache* c, int64_t x) {
  int64_t cnt;
  int64_t y = tier_first_out(c, CKVO_TIER_CPU, &cnt);
  if (cnt < c->cpu_slots) {
    c->tier[x] = CKVO_TIER_CPU;
    return 1;
  }
  if (y >= 0 && leaves_before(c, y, x)) {
    c->tier[y] = CKVO_TIER_NONE;
    c->counts.dropped++;
    c->tier[x] = CKVO_TIER_CPU;
    return 1;
  }
  c->tier[x] = CKVO_TIER_NONE;
  c->counts.dropped++;
  return 0;
}

/* Places x in the GPU tier if there is room or x outranks the GPU tier's
 * weakest entry, which then goes down to the CPU tier (or out of memory);
 * otherwise x itself goes to the CPU tier. */
static void admit_gpu(ckvo_cache* c, int64_t x) {
  int64_t cnt;
  int64_t y = tier_first_out(c, CKVO_TIER_GPU, &cnt);
  if (cnt < c->gpu_slots) {
    c->tier[x] = CKVO_TIER_GPU;
    return;
  }
  if (y >= 0 && leaves_before(c, y, x)) {
    c->tier[y] = CKVO_TIER_NONE;
    c->tier[x] = CKVO_TIER_GPU;
    c->counts.demoted += admit_cpu(c, y);
    return;
  }
  admit_cpu(c, x);
}

/* Sec. 4.5: for each used chunk in order, note where it was found, add its
 * attention score to I and one access to F, then re-place it by its new
 * cache score: GPU tier first, then CPU tier, evicting the weakest entries. */
int ckvo_cache_access(ckvo_cache* c, const int64_t* keys, const double* A, int64_t count,
                      int8_t* tier_before, ckvo_cache_counts* counts) {
  if (!c || count < 0 || (count > 0 && (!keys || !A))) return -1;
  for (int64_t u = 0; u < count; ++u) {
    if (keys[u] < 0 || keys[u] >= c->n_keys || !(A[u] >= 0.0) || A[u] > DBL_MAX) return -1;
    for (int64_t v = 0; v < u; ++v)
      if (keys[v] == keys[u]) return -1;
  }
  for (int64_t u = 0; u < count; ++u) {
    int64_t x = keys[u];
    int8_t was = c->tier[x];
    if (tier_before) tier_before[u] = was;
    if (was == CKVO_TIER_GPU) c->counts.hits_gpu++;
    else if (was == CKVO_TIER_CPU) c->counts.hits_cpu++;
    else c->counts.misses++;
    c->I[x] += A[u];
    /* F: every use; or, read literally, every load into GPU or CPU memory
     * (a use of a chunk already in the GPU tier loads nothing) */
    if (c->policy != CKVO_CACHE_LOADS || was != CKVO_TIER_GPU) c->F[x] += 1;
    c->last[x] = ++c->clock;
    c->tier[x] = CKVO_TIER_NONE;
    admit_gpu(c, x);
  }
  if (counts) *counts = c->counts;
  return 0;
}

int ckvo_cache_state(const ckvo_cache* c, double* I, int64_t* F, int8_t* tier) {
  if (!c) return -1;
  for (int64_t x = 0; x < c->n_keys; ++x) {
    if (I) I[x] = c->I[x];
    if (F) F[x] = c->F[x];
    if (tier) tier[x] = c->tier[x];
  }
  return 0;
}
