/*
 * ckv_oracle.h -- CPU oracle for the ContiguousKV Re-Prefill hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  This is the plain, slow, fp64 reference that the
 * GPU library is checked against.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load it; the product path never does.  It
 * shares no code, header, table or helper with the GPU library.
 *
 * Paper: "ContiguousKV: Accelerating LLM Prefill with Granularity-Aligned KV
 * Cache Management" (arXiv 2601.13631).  Every function cites the passage it
 * follows.  Where the paper is silent or garbled the reading taken is stated at
 * the function.
 *
 * Tensor layouts (all row-major, contiguous, host memory):
 *   q          [S][Hq][d]      suffix queries
 *   k_prefix   [n][Hkv][d]     stored prefix keys
 *   v_prefix   [n][Hkv][d]     stored prefix values
 *   k_suffix   [S][Hkv][d]     suffix keys
 *   v_suffix   [S][Hkv][d]     suffix values
 *   out        [S][Hq][d]      fp64 attention output
 * Element type of the inputs: CKVO_F32 (float) or CKVO_BF16 (uint16 bf16 bit
 * patterns); both are widened exactly to double before any arithmetic.
 *
 * Return value of every int-returning function: 0 on success, -1 on invalid
 * arguments (nothing is written), -2 on allocation failure.
 */
#ifndef CKV_ORACLE_H
#define CKV_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { CKVO_F32 = 0, CKVO_BF16 = 1 };

typedef struct {
  int64_t n_prefix;   /* n: prefix tokens                      */
  int32_t n_suffix;   /* S: suffix tokens (queries)             */
  int32_t n_q_heads;  /* Hq                                     */
  int32_t n_kv_heads; /* Hkv; Hq % Hkv == 0 (GQA group G=Hq/Hkv) */
  int32_t head_dim;   /* d                                      */
  int32_t chunk_size; /* c: tokens per ContiguousChunk          */
  int32_t dtype;      /* CKVO_F32 or CKVO_BF16                  */
  double sm_scale;    /* logit scale; 0 selects 1/sqrt(d)       */
} ckvo_shape;

/* Def. 4.1: m = ceil(n / c).  Returns -1 for n < 0 or c < 1. */
int64_t ckvo_num_chunks(int64_t n, int32_t c);

/* Number of chunks kept at budget ratio r (paper silent on rounding):
 * k = clamp(ceil(r*m - 1e-9), 1, m); 0 when m == 0; -1 when r is not in (0,1]. */
int64_t ckvo_num_keep(int64_t m, double r);

/* Sec. 4.4 token importance: a[i] = sum over every suffix query t and every
 * query head h of softmax_i(sm_scale * q[t,h] . k[i, h/G]) over the n prefix
 * keys.  a has n entries.  nthreads <= 0 uses all online CPUs.  The result does
 * not depend on nthreads. */
int ckvo_token_importance(const ckvo_shape* s, const void* q, const void* k_prefix,
                          double* a, int nthreads);

/* Eq. 1 sum pooling: A[j] = sum of a[i] over the tokens of chunk j, ascending. */
int ckvo_chunk_scores(const ckvo_shape* s, const double* a, double* A);

/* Top-k chunk selection under the total order (score descending, index
 * ascending); NaN ranks below every number and -0.0 equals +0.0.  Writes the k
 * chosen chunk indices to sel in ascending order.  Requires 1 <= k <= m. */
int ckvo_select_topk(const double* A, int64_t m, int64_t k, int32_t* sel);

/* Def. 2.1 re-prefill attention over the selected prefix chunks plus the
 * causal suffix.  For query t and head h the key sequence is the tokens of
 * every selected chunk (sel ascending, each chunk's tokens ascending) followed
 * by suffix tokens 0..t.  out_rows selects which (t, h) outputs to compute:
 * NULL computes all S*Hq rows into out[S][Hq][d]; otherwise row_ids[r] = t*Hq+h
 * for r < n_rows and out is [n_rows][d].  sel must be strictly ascending and
 * inside [0, m). */
int ckvo_sparse_attn(const ckvo_shape* s, const void* q, const void* k_prefix,
                     const void* v_prefix, const int32_t* sel, int64_t k,
                     const void* k_suffix, const void* v_suffix,
                     const int64_t* row_ids, int64_t n_rows, double* out, int nthreads);

/* Dense re-prefill attention: every prefix token, then the causal suffix.
 * Written as its own loop; with every chunk selected it visits the same keys in
 * the same order as ckvo_sparse_attn and so agrees with it bit for bit. */
int ckvo_dense_attn(const ckvo_shape* s, const void* q, const void* k_prefix,
                    const void* v_prefix, const void* k_suffix, const void* v_suffix,
                    const int64_t* row_ids, int64_t n_rows, double* out, int nthreads);

/* Contiguous gather (Sec. 4.2): copies the K and V spans of every selected
 * chunk into compact [k*c][Hkv][d] buffers; rows past n in a partial last chunk
 * are zero.  Byte copy, no arithmetic. */
int ckvo_gather_chunks(const ckvo_shape* s, const void* k_src, const void* v_src,
                       const int32_t* sel, int64_t k, void* k_dst, void* v_dst);

/* Prefetch accounting of Sec. 4.3.2 with the previous layer's set as the
 * prediction.  sel (k, ascending) is this layer's set, pred (n_pred, ascending,
 * may be empty) the prefetched one.  span(j) = 2 * |chunk j| * Hkv * d * elem
 * bytes (K span plus V span). */
typedef struct {
  int64_t k, hits, misses, wasted;
  int64_t bytes_prefetch, bytes_demand, bytes_used;
} ckvo_layer_stats;
int ckvo_layer_accounting(const ckvo_shape* s, const int32_t* sel, int64_t k,
                          const int32_t* pred, int64_t n_pred, ckvo_layer_stats* st);

/* Read accounting (Sec. 4.2; Sec. 3, Motivation 1).  A ContiguousChunk store
 * reads exactly the tokens of the selected chunks; a store cut into fixed
 * blocks of b consecutive tokens (the comparison systems use 64) reads every
 * block that holds at least one of them.  sel holds k distinct chunk indices in
 * [0, ceil(n/c)), any order.  Counts:
 *   tokens_selected  tokens of the selected chunks (the last chunk clamped to n)
 *   runs             maximal runs of consecutive selected chunks
 *   blocks           blocks holding a selected token
 *   tokens_block     tokens in those blocks (the last block clamped to n) */
typedef struct {
  int64_t tokens_selected, runs, blocks, tokens_block;
} ckvo_io_counts;
int ckvo_io_account(int64_t n, int32_t c, const int32_t* sel, int64_t k, int32_t b,
                    ckvo_io_counts* out);

/* Attention-guided cache management (Sec. 4.5, Eq. 2).  Keys 0..n_keys-1 name
 * cacheable ContiguousChunks.  Every key keeps I (sum of the attention scores A
 * of its accesses), F (number of accesses) and the time of its latest access,
 * for evicted keys too (the in-memory score table).  Two tiers of gpu_slots and
 * cpu_slots entries hold keys by cache score S = I*F (policy ATTENTION) or S = F
 * (policy LFU, the ablation's frequency-only foil).  Policy LOADS is S = I*F
 * with F read literally as the number of times the chunk was loaded into GPU
 * or CPU memory: a use of a key already in the GPU tier adds to I but not to
 * F.  Readings where the paper is silent: F counts accesses (ATTENTION, LFU);
 * an accessed key goes to the GPU tier when there
 * is room or it outranks the GPU tier's weakest entry, which is then demoted to
 * the CPU tier by the same rule, else the key goes to the CPU tier by that
 * rule; whatever the CPU tier does not take leaves memory; ranking is by S,
 * then by latest access (older leaves first).  This oracle finds the weakest
 * entry by scanning every key. */
enum { CKVO_CACHE_ATTENTION = 0, CKVO_CACHE_LFU = 1, CKVO_CACHE_LOADS = 2 };
enum { CKVO_TIER_NONE = 0, CKVO_TIER_CPU = 1, CKVO_TIER_GPU = 2 };
typedef struct {
  int64_t hits_gpu, hits_cpu, misses; /* where each accessed key was found        */
  int64_t demoted;                    /* GPU-tier evictions taken by the CPU tier  */
  int64_t dropped;                    /* keys that left memory (or never entered)  */
} ckvo_cache_counts;
typedef struct ckvo_cache ckvo_cache;
ckvo_cache* ckvo_cache_create(int64_t n_keys, int64_t gpu_slots, int64_t cpu_slots, int policy);
void ckvo_cache_destroy(ckvo_cache* c);
/* One request's used chunks: keys[count] distinct, A[count] finite and >= 0,
 * processed in the given order.  tier_before[u] (may be NULL) receives where
 * keys[u] was found; *counts (may be NULL) the totals since creation. */
int ckvo_cache_access(ckvo_cache* c, const int64_t* keys, const double* A, int64_t count,
                      int8_t* tier_before, ckvo_cache_counts* counts);
/* Copies I, F and tier of every key (each pointer may be NULL). */
int ckvo_cache_state(const ckvo_cache* c, double* I, int64_t* F, int8_t* tier);

/* One Re-Prefill layer of the hot path: token importance, Eq. 1 pooling,
 * top-k at keep ratio r, sparse attention.  Writes A[m], sel[k] and out[S][Hq][d];
 * *k_out receives k. */
int ckvo_reprefill_layer(const ckvo_shape* s, double keep_ratio, const void* q,
                         const void* k_prefix, const void* v_prefix, const void* k_suffix,
                         const void* v_suffix, double* A, int32_t* sel, int64_t* k_out,
                         double* out, int nthreads);

#ifdef __cplusplus
}
#endif
#endif
