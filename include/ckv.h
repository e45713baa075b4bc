/*
 * ckv.h -- C ABI of libckv, the MI355X (gfx950) implementation of the
 * data-parallel hot path of ContiguousKV's Re-Prefill phase.
 *
 * Paper: "ContiguousKV: Accelerating LLM Prefill with Granularity-Aligned KV
 * Cache Management", arXiv 2601.13631.  For one transformer layer the path
 *   1. scores every prefix key against the new suffix's queries and sums the
 *      softmax probabilities per ContiguousChunk           (Sec. 4.4, Eq. 1)
 *   2. keeps the k highest-scoring chunks                   (Sec. 4.4; Sec. 5.1 budgets)
 *   3. moves only those chunks' contiguous K/V spans        (Sec. 4.2)
 *      -- from HBM, or from pinned host memory with the next layer's chunks
 *         prefetched from this layer's set                   (Sec. 4.3.2)
 *   4. runs the suffix's attention over the kept prefix KV plus the causal
 *      suffix KV                                            (Def. 2.1)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Return value: a ckv_status.  Arguments are validated before anything is
 *   launched; on an error nothing has been enqueued and no output is touched.
 *   No entry point aborts, exits or throws.  ckv_last_error() returns a
 *   thread-local text describing the most recent failure on this thread.
 * - Ownership: the caller owns every buffer passed in.  The library never
 *   frees, retains or reallocates caller memory.
 * - Device pointers must point to memory of the current HIP device; tensor base
 *   pointers must be 16-byte aligned.
 * - Asynchrony: work is enqueued on the caller's stream (a hipStream_t passed
 *   as void*; NULL is the null stream).  Outputs are valid once that stream has
 *   been synchronized.  Inputs must stay valid and unchanged until then.
 * - Scratch memory comes from a caller-provided workspace (device memory of at
 *   least the size the matching *_workspace_bytes() call returns, 256-byte
 *   aligned), or from a ckv_ctx.
 * - Thread safety: entry points without a ckv_ctx are reentrant; a ckv_ctx
 *   must be used by one host thread at a time.
 *
 * Tensor layouts (row-major, contiguous; element type from ckv_dims.dtype)
 * ------------------------------------------------------------------------
 *   q            [S][Hq][d]    suffix queries (post-RoPE)
 *   k_prefix     [n][Hkv][d]   stored prefix keys;   chunk j = rows [j*c, min(j*c+c, n))
 *   v_prefix     [n][Hkv][d]   stored prefix values
 *   k_suffix     [S][Hkv][d]   suffix keys
 *   v_suffix     [S][Hkv][d]   suffix values
 *   k_sel, v_sel [k*c][Hkv][d] gathered chunks, chunk u at rows [u*c, u*c+c)
 *   out          [S][Hq][d]    attention output, same element type as q
 * With this layout one ContiguousChunk of one tensor is a single contiguous
 * span of c*Hkv*d elements (Sec. 4.2: the chunk is the unit of storage and I/O).
 * Query head h reads KV head h / (Hq/Hkv) (grouped-query attention, Sec. 2.1).
 */
#ifndef CKV_H
#define CKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t ckv_status;
#define CKV_OK 0
#define CKV_EINVAL 1         /* bad shape, pointer, alignment or size */
#define CKV_EUNSUPPORTED 2   /* valid but not built: dtype/head_dim/chunk_size combination */
#define CKV_EHIP 3           /* a HIP runtime call failed; see ckv_last_error() */
#define CKV_ENOMEM 4         /* device or pinned host allocation failed */
#define CKV_ESTATE 5         /* ckv_ctx used out of order */

#define CKV_DTYPE_F32 0
#define CKV_DTYPE_BF16 1

/* Problem shape.  Supported: dtype BF16 with head_dim 64 or 128, dtype F32
 * with head_dim 64; chunk_size 4, 8, 16 or a multiple of 32; n_prefix >= 1;
 * n_suffix >= 1; n_q_heads a multiple of n_kv_heads. */
typedef struct ckv_dims {
  int64_t n_prefix;   /* n: prefix tokens                             */
  int32_t n_suffix;   /* S: suffix tokens (queries)                    */
  int32_t n_q_heads;  /* Hq                                            */
  int32_t n_kv_heads; /* Hkv                                           */
  int32_t head_dim;   /* d                                             */
  int32_t chunk_size; /* c: tokens per ContiguousChunk (Def. 4.1)       */
  int32_t dtype;      /* CKV_DTYPE_F32 or CKV_DTYPE_BF16               */
  float sm_scale;     /* logit scale; 0 selects 1/sqrt(head_dim)       */
} ckv_dims;

/* Thread-local text of the last failure on this thread ("" if none). */
const char* ckv_last_error(void);

/* Library version string. */
const char* ckv_version(void);

/* Def. 4.1: number of ContiguousChunks m = ceil(n / c).  -1 if n < 0 or c < 1.
 * Host-only, pure. */
int64_t ckv_num_chunks(int64_t n, int32_t c);

/* Chunks kept at budget ratio r in (0, 1] (the evaluation's KV budget ratios,
 * Sec. 5.1; the paper does not fix the rounding):
 * k = clamp(ceil(r*m - 1e-9), 1, m), 0 when m == 0, -1 when r is outside
 * (0, 1] or m < 0.  Host-only, pure, so a caller knows k without a device sync. */
int64_t ckv_num_keep(int64_t m, double r);

/* ---------------------------------------------------------------------------
 * Chunk scoring -- Sec. 4.4 and Eq. 1.
 * For every query head h and suffix query t, the probabilities
 * softmax_i(sm_scale * q[t,h] . k_prefix[i, h/G]) over the n prefix keys are
 * summed per chunk and over all (t, h):
 *   chunk_scores[j] = sum_{t,h} sum_{i in chunk j} p_{t,h,i}.
 * The softmax runs over the prefix keys only, so sum_j chunk_scores[j] = S*Hq.
 *   q             device, [S][Hq][d]
 *   k_prefix      device, [n][Hkv][d]
 *   chunk_scores  device, double[m] (written)
 *   ws            device workspace of ckv_score_workspace_bytes(dims) bytes
 *                 (0 for a shape too large for the scoring decomposition);
 *                 scratch, no initial contents needed.  Calls that share a
 *                 workspace must not overlap in time.
 * Arithmetic: logits and exponentials in fp32 (bf16 products are exact in
 * fp32), per-chunk partial sums in fp32 over at most one chunk, every sum
 * across rows, key segments and heads in fp64, in a fixed order (run-to-run
 * deterministic).
 * ------------------------------------------------------------------------- */
size_t ckv_score_workspace_bytes(const ckv_dims* dims);
ckv_status ckv_score_chunks(const ckv_dims* dims, const void* q, const void* k_prefix,
                            double* chunk_scores, void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Top-k chunk selection -- Sec. 4.4 (chunks ranked by A_j, the k highest
 * kept), budgets of Sec. 5.1.
 * Keeps the k largest scores under the total order (score descending, index
 * ascending): among equal scores the lower chunk index wins.  -0.0 equals
 * +0.0; NaN ranks below every number.  Writes the k chosen indices in
 * ascending order.  Bit-exact: the result depends only on the score bits.
 *   chunk_scores  device, double[m]
 *   sel_idx       device, int32[k] (written)
 *   1 <= k <= m <= 2^31-1
 * ------------------------------------------------------------------------- */
size_t ckv_select_workspace_bytes(int64_t m);
ckv_status ckv_select_topk_chunks(const double* chunk_scores, int64_t m, int64_t k,
                                  int32_t* sel_idx, void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Contiguous chunk gather -- Sec. 4.2 (only the selected chunks move, each as
 * whole contiguous spans: no block read amplification).
 * Copies the K and V spans of chunks sel_idx[0..k) into k_sel / v_sel,
 * chunk u to rows [u*c, u*c+c); rows past n of a short last chunk are zeroed.
 *   k_src, v_src  [n][Hkv][d], device memory or pinned host memory mapped
 *                 into the device address space (hipHostMalloc); pageable
 *                 host memory is refused with CKV_EINVAL
 *   sel_idx       device, int32[k], each in [0, m) (indices are not checked on
 *                 the host; an index outside [0, m) is clamped by the kernel
 *                 and its span is zero-filled)
 *   k_sel, v_sel  device, [k*c][Hkv][d] (written)
 * ------------------------------------------------------------------------- */
ckv_status ckv_gather_chunks(const ckv_dims* dims, const void* k_src, const void* v_src,
                             const int32_t* sel_idx, int64_t k, void* k_sel, void* v_sel,
                             void* stream);

/* ---------------------------------------------------------------------------
 * Re-Prefill sparse attention -- Def. 2.1 (the suffix attends over the loaded
 * prefix KV and its own KV), GQA of Sec. 2.1.
 * For query t of head h the keys are the tokens of the k gathered chunks (in
 * order; rows past n of a short last chunk skipped) followed by suffix tokens
 * 0..t (causal).  out[t][h] = sum softmax(sm_scale * q.k) * v; softmax in
 * fp32 with bf16 MFMA products for bf16 inputs.
 *   q             device, [S][Hq][d]
 *   k_sel, v_sel  device, [k*c][Hkv][d] (as written by ckv_gather_chunks)
 *   sel_idx       device, int32[k]: the chunks' indices, used only to find the
 *                 length of a short last chunk
 *   k_suffix, v_suffix  device, [S][Hkv][d]
 *   out           device, [S][Hq][d] (written)
 *   ws            device workspace of ckv_attn_workspace_bytes(dims, k) bytes
 * 0 <= k <= m.  Inputs must be finite: the bf16 kernel is built without NaN
 * semantics, so a NaN in Q, K or V gives unspecified output.
 * ------------------------------------------------------------------------- */
size_t ckv_attn_workspace_bytes(const ckv_dims* dims, int64_t k);
ckv_status ckv_sparse_prefill_attn(const ckv_dims* dims, const void* q, const void* k_sel,
                                   const void* v_sel, const int32_t* sel_idx, int64_t k,
                                   const void* k_suffix, const void* v_suffix, void* out,
                                   void* ws, size_t ws_bytes, void* stream);

/* Test hook for the attention's K/V addressing.  A source whose rows all lie
 * below 4 GiB from its base is read through 32-bit byte offsets; a larger one
 * through a 64-bit address per row.  force_wide = 1 makes every later launch
 * in the process (standalone or in a layer step) take the 64-bit form, so that
 * tests can run it on small inputs; the two forms read the same bytes and give
 * bit-identical results.  0 restores the default.  Process-wide, thread-safe;
 * launches already enqueued are not affected. */
ckv_status ckv_debug_attn_wide_addressing(int32_t force_wide);

/* ---------------------------------------------------------------------------
 * Layer step -- one Re-Prefill layer: score -> select -> move chunks ->
 * attention, with the context owning streams, events, workspace and (for a
 * host-resident prefix) HBM chunk slots.
 * ------------------------------------------------------------------------- */
typedef struct ckv_ctx ckv_ctx;
typedef struct ckv_cache ckv_cache; /* Sec. 4.5 cache, see ckv_cache_create */
typedef struct ckv_store ckv_store; /* storage tier, see ckv_store_open */

/* ctx flags */
#define CKV_CTX_HOST_PREFIX 0x1     /* prefix K/V live in pinned host memory (Sec. 4.3.2) */
#define CKV_CTX_MATERIALIZE 0x2     /* HBM prefix: gather into compact buffers before
                                       attention instead of reading spans in place */
#define CKV_CTX_STAGE_TIMING 0x4    /* record HIP events between the stages of every
                                       layer (see ckv_ctx_stage_times) */
#define CKV_CTX_SCORE_TIMING 0x8    /* time only the chunk-scoring main kernel and
                                       nothing else (bf16: from its first workgroup's
                                       start to its last workgroup's end, stamped by
                                       the kernel from the 100 MHz realtime counter,
                                       so no event sits between the launches; fp32:
                                       two events per layer);
                                       ckv_ctx_stage_times then reports the score stage
                                       and zero for the others */

/* Stages timed with CKV_CTX_STAGE_TIMING. */
#define CKV_STAGE_SCORE 0     /* chunk-scoring main kernel                         */
#define CKV_STAGE_FINALIZE 1  /* fp64 fold of the partial sums into chunk scores   */
#define CKV_STAGE_SELECT 2    /* top-k selection                                   */
#define CKV_STAGE_MOVE 3      /* gather, or the wait for demand copies (host prefix) */
#define CKV_STAGE_ATTN 4      /* attention (and split combine)                     */
#define CKV_N_STAGES 5

/* Creates a context for layers 0 .. n_layers-1 of shape *dims at keep ratio
 * keep_ratio.  Allocates the workspace (and, with CKV_CTX_HOST_PREFIX, a ring
 * of HBM slot buffers of 2k chunks each plus pinned index staging) on the
 * current device.  *out receives the context.  CKV_EINVAL for n_layers < 1 or
 * keep_ratio outside (0, 1]. */
ckv_status ckv_ctx_create(const ckv_dims* dims, int32_t n_layers, double keep_ratio, int32_t flags,
                          ckv_ctx** out);
/* Waits for the context's streams, then frees everything the context owns. */
ckv_status ckv_ctx_destroy(ckv_ctx* ctx);
/* Starts a request over: forgets the previous layer's selection and every
 * prediction (the next layer, which may be any layer, runs as the first of a
 * request), the set held for the current Period, the stage times, an armed
 * copy-error injection, and the failed state a layer error leaves.  Waits for
 * the context's copy streams. */
ckv_status ckv_ctx_reset(ckv_ctx* ctx);

/* Periods -- Def. 4.2 (Sec. 4.3): consecutive layers p*i .. p*i+p-1 form a
 * Period and share one important-chunk set, the one selected at layer p*i.
 * With period p > 1, ckv_reprefill_layer runs scoring and selection only on
 * a layer that is a multiple of p and keeps the set in the context; every
 * other layer attends over the set of its Period's first layer, which must
 * have run on this context since the last reset or set_period (else
 * CKV_ESTATE), writes that set to io->sel_idx (if given), leaves
 * io->chunk_scores untouched, and needs no host synchronisation even with a
 * host-resident prefix (its prefetch prediction, the previous layer's set,
 * is then exact).  period = 1 (the default) selects at every layer.
 * With a host-resident prefix whose per-layer stores are registered
 * (ckv_ctx_set_host_layers), no store attached and 1 < p <= 16, a Period's
 * first layer also queues the copies of every later layer of its Period
 * (intra-period prefetch, Sec. 4.3.2) as soon as its set is known; the HBM
 * ring then holds p + 1 buffers of 2k chunk slots.  Then the Period must be
 * set at the start of a request (CKV_ESTATE otherwise; it synchronizes the
 * device when the ring changes).  Forgets any set held.  CKV_EINVAL if
 * period < 1. */
ckv_status ckv_ctx_set_period(ckv_ctx* ctx, int32_t period);

/* Attention-guided cache on the layer step -- Sec. 4.5 (with the cache of
 * ckv_cache_create).  Attaches `cache` to a context with a host-resident
 * prefix (CKV_CTX_HOST_PREFIX), or detaches the current one (cache NULL).
 * The context then keeps the chunks of the cache's GPU tier in
 * min(gpu_slots, n_keys) HBM chunk slots that it allocates here (each slot
 * one chunk's K span and V span), key = layer * m + chunk, so the cache's
 * n_keys must be a multiple of m and layers beyond n_keys / m are refused.
 * Each host-resident layer then
 *   - reads the selected chunks held in those slots in place (stats
 *     cache_hits): no host-link copy;
 *   - prefetches and fetches on demand only the other chunks;
 *   - after its attention, calls ckv_cache_access with its chunks and their
 *     scores A_j (for a layer inside a Period, those of the Period's first
 *     layer) and copies each chunk that entered the GPU tier from its
 *     transient slot into a cache slot (stats bytes_cache_fill); chunks that
 *     left the GPU tier free their slots (their bytes stay in the host store).
 * The cache persists across requests (ckv_ctx_reset keeps it), so later
 * requests on the same prefix find its heavily used chunks in HBM.  Every
 * request must pass the same per-layer kv_host contents while it is
 * attached.  Must be called before a request's first layer (or after
 * ckv_ctx_reset), else CKV_ESTATE; the cache's GPU tier must be empty
 * (CKV_ESTATE); with a store attached (ckv_ctx_attach_store) it is refused
 * (CKV_ESTATE): attach the cache first, since the store's chunk pool is sized
 * for the cache's tiers.  Synchronizes the device.  The context does not own the
 * cache: detach it (or destroy the context) before destroying it or calling
 * ckv_cache_access on it directly.  With a cache attached, a layer inside a
 * Period waits on the host for the copies two layers back before it reuses
 * their staging buffers. */
ckv_status ckv_ctx_attach_cache(ckv_ctx* ctx, ckv_cache* cache);

/* Storage tier on the layer step (with a store of ckv_store_open whose
 * span_bytes is one chunk's K and V spans and whose n_keys is a multiple of m:
 * key = layer * m + chunk).  Attaches `store` to a context with a
 * host-resident prefix, or detaches it (NULL).  The context then allocates two
 * pinned staging buffers of 2k chunks and takes every chunk a layer moves to
 * HBM from the file instead of from io->kv_host (which may be NULL;
 * kv_host_next is ignored), through a pinned chunk pool that it allocates:
 *   - the chunks a layer fetches on demand that are not in the pool are read
 *     by the I/O threads into free pool slots (the layer waits for them), then
 *     copied to HBM;
 *   - the prediction for layer + 1 (this layer's set less the chunks the next
 *     layer finds in an attached cache's HBM slots) is read asynchronously,
 *     where not in the pool, while this layer attends, and copied to HBM at
 *     the start of layer + 1, beside its scoring;
 *   - with a cache attached, the pool keeps the chunks of the cache's GPU and
 *     CPU tiers (min(gpu_slots + cpu_slots, n_keys) of them, plus room for two
 *     layers in flight): a chunk in the CPU tier is copied from host memory
 *     without a file read, as Sec. 4.5's CPU heap intends; every other pool
 *     slot is released after its layer and reused one layer later;
 *   - layers past n_keys / m are refused (CKV_EINVAL).
 * Stats bytes_prefetch and bytes_demand count bytes moved to HBM over the
 * host link as before; bytes_storage counts the bytes read from the file.
 * Same call rules as ckv_ctx_attach_cache (start of a request, synchronizes
 * the device); attach a cache before the store and detach the store before
 * the cache; detach or destroy the context before closing the store.  With a store attached, ckv_ctx_reset synchronizes
 * the device, and a layer inside a Period waits on the host for the previous
 * layer's attention before it reuses pool slots. */
ckv_status ckv_ctx_attach_store(ckv_ctx* ctx, ckv_store* store);

/* SubPeriod -- the SubPeriod size of the evaluation setup with Sec. 4.3.2's
 * intra-period prefetch (and Def. 4.2's Periods).
 *   - Pinned-host prefix with intra-period prefetch (see ckv_ctx_set_period):
 *     the attention of a Period's first layer starts only once the chunks of
 *     the Period's first `subperiod` layers (its own included) are in HBM:
 *     the gate that decides how many layers' KV must be loaded before the
 *     Period's computation begins.  subperiod = 1 gates nothing beyond each
 *     layer's own chunks.
 *   - Storage tier (a store attached) with a Period of p > 1 layers: a layer
 *     queues the storage reads of every later layer of its Period up to
 *     subperiod - 1 layers ahead as soon as its set is known (the set is the
 *     Period's, so these predictions are exact); a layer's computation waits
 *     only for its own chunks.  subperiod = 1 reads one layer ahead.
 * 1 <= subperiod <= 16 (CKV_EINVAL); must be set before the store is attached
 * (CKV_ESTATE), since it sizes the chunk pool (subperiod * k more slots).
 * Gating only orders work: results do not depend on it. */
ckv_status ckv_ctx_set_subperiod(ckv_ctx* ctx, int32_t subperiod);

/* Registers the pinned host stores of every layer (kv_host[l] for layer l, in
 * ckv_layer_io.kv_host's layout; n == n_layers) with a host-resident context,
 * or unregisters them (kv_host NULL).  Layers may then pass io->kv_host and
 * io->kv_host_next as NULL (the registered stores are used; if io->kv_host is
 * given it is used for the layer's own chunks), and a Period's first layer
 * can queue the copies of the whole Period (intra-period prefetch, see
 * ckv_ctx_set_period).  The stores must stay valid and unchanged while
 * registered.  At the start of a request only (CKV_ESTATE); CKV_EINVAL for a
 * count that is not n_layers or a store that is not pinned host memory
 * (nothing changes then).  Ignored while a store is attached. */
ckv_status ckv_ctx_set_host_layers(ckv_ctx* ctx, const void* const* kv_host, int32_t n);

/* Test hook for failure handling: the next run of `layer` on this
 * host-resident context fails where it would enqueue its host-to-HBM demand
 * copies, as if that copy had failed: ckv_reprefill_layer returns CKV_EHIP
 * (after its scoring and selection were enqueued, none of its copies or its
 * attention), and the context refuses layers until ckv_ctx_reset.  layer = -1
 * disarms; a reset disarms too.  CKV_EINVAL for an HBM-resident context or a
 * layer outside [-1, n_layers). */
ckv_status ckv_ctx_inject_copy_error(ckv_ctx* ctx, int32_t layer);

typedef struct ckv_layer_io {
  const void* q;         /* device [S][Hq][d]                                        */
  const void* k_suffix;  /* device [S][Hkv][d]                                       */
  const void* v_suffix;  /* device [S][Hkv][d]                                       */
  const void* k_probe;   /* device [n][Hkv][d]: the layer's prefix keys for scoring  */
  const void* k_prefix;  /* device [n][Hkv][d] (HBM-resident prefix), else NULL      */
  const void* v_prefix;  /* device [n][Hkv][d] (HBM-resident prefix), else NULL      */
  const void* kv_host;   /* pinned host (hipHostMalloc; pageable memory is refused),
                            chunk-major: chunk j of this layer at byte offset
                            j * 2*c*Hkv*d*elem, K span then V span; rows past n of
                            the last chunk are padding (host-resident prefix); may
                            be NULL when the stores are registered
                            (ckv_ctx_set_host_layers)                               */
  const void* kv_host_next; /* the next layer's kv_host, prefetched during this layer
                               with this layer's selection as the prediction; NULL
                               for the last layer (or no prefetch); ignored when the
                               stores are registered                                 */
  void* out;             /* device [S][Hq][d] (written)                              */
  double* chunk_scores;  /* device double[m] (written), or NULL                      */
  int32_t* sel_idx;      /* device int32[k] (written), or NULL                       */
  void* stream;          /* hipStream_t for the layer's compute                      */
  const int32_t* pred_idx; /* host int32[n_pred], strictly ascending chunk indices: this
                              layer's predicted set (Sec. 4.3.2: the chunks expected
                              to be selected, e.g. the previous Period's or layer's
                              set), copied to HBM beside this layer's scoring; it
                              replaces the context's own prediction.  NULL: the
                              context's own (the previous layer's set, when the
                              previous call ran layer - 1 with a next store).
                              Host-resident prefix only (ignored, but validated,
                              for an HBM-resident one); not with a store attached
                              (CKV_EUNSUPPORTED)                                     */
  int64_t n_pred;        /* entries of pred_idx, 0 <= n_pred <= k (0: an empty
                              prediction, every kept chunk fetched on demand)        */
} ckv_layer_io;

typedef struct ckv_layer_stats {
  int64_t k;               /* chunks selected                                         */
  int64_t hits;            /* selected chunks that were prefetched                     */
  int64_t misses;          /* selected chunks fetched on demand                        */
  int64_t wasted;          /* prefetched chunks not selected                           */
  int64_t bytes_prefetch;  /* host->HBM bytes issued for the next layer's prediction   */
  int64_t bytes_demand;    /* host->HBM bytes fetched on demand for this layer         */
  int64_t bytes_gathered;  /* K+V bytes of the selected chunks (= bytes attended); with
                              an HBM-resident prefix the set stays on the device and a
                              kept short last chunk is counted at full length          */
  int64_t cache_hits;      /* selected chunks read from an attached cache's HBM slots
                              (no host-link transfer; not counted in hits or misses)   */
  int64_t bytes_cache_fill;/* HBM->HBM bytes copied into cache slots for chunks that
                              entered the cache's GPU tier at this layer (whole slots) */
  int64_t bytes_storage;   /* bytes read from an attached store at this layer (demand
                              reads plus the next layer's prediction; whole spans)     */
} ckv_layer_stats;

/* Sum of the GPU time of each stage (ms[CKV_N_STAGES], milliseconds) over
 * every layer run since the context was created or last reset, and that
 * number of layers in *n_layers.  Requires CKV_CTX_STAGE_TIMING or
 * CKV_CTX_SCORE_TIMING (then only ms[CKV_STAGE_SCORE] is filled, and only
 * layers that ran scoring are counted); waits for the layers not yet
 * accounted (with CKV_CTX_SCORE_TIMING on bf16, for the whole device).  Stage
 * times come from events recorded on each layer's compute stream between its
 * kernel launches, or, for the bf16 scoring kernel alone, from the kernel's
 * own timestamps. */
ckv_status ckv_ctx_stage_times(ckv_ctx* ctx, double* ms, int64_t* n_layers);

/* Runs layer `layer` (0 <= layer < n_layers; the first layer after creation
 * or ckv_ctx_reset may be any layer and has no prediction unless io gives
 * one).  HBM-resident prefix: returns without a host synchronization.
 * Host-resident prefix: synchronizes once on the selection (the only
 * device->host dependency of the step), enqueues the demand copies of the
 * missed chunks, the attention over the HBM slots and the prefetch of the
 * next layer's chunks.  With bf16 the attention runs in parts over the same
 * kept set -- the chunks already in HBM (prefetched or in a cache's slots)
 * with the suffix during the demand copies, then each share of the missed
 * chunks once it has landed -- merged in a fixed order: the output is
 * deterministic, but it is bit-identical to another context's only when the
 * same chunks were already in HBM.  Counts in *stats (may be NULL) are exact; after the
 * first layer of a request, layers must run in order (layer + 1, else
 * CKV_ESTATE).  If the call fails after it has enqueued work (a HIP error,
 * an injected copy error), the context refuses further layers with
 * CKV_ESTATE until ckv_ctx_reset, after which it is fully usable. */
ckv_status ckv_reprefill_layer(ckv_ctx* ctx, int32_t layer, const ckv_layer_io* io,
                               ckv_layer_stats* stats);

/* ---------------------------------------------------------------------------
 * The layer step without allocation -- for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  One HBM-resident layer (score -> select ->
 * attention over the kept chunks' spans read in place) like ckv_reprefill_layer
 * on an HBM-resident context, with the same kernels and bit-identical results,
 * but with no context: its scratch is a fixed device array of
 * CKV_NOALLOC_SCRATCH_BYTES inside the library (each device the library runs
 * on holds its own copy until the process ends; its address is looked up on a
 * device's first call).  The call allocates nothing and needs no initial
 * scratch contents.  Scratch needed: max(ckv_score_workspace_bytes,
 * ckv_attn_workspace_bytes(k)) rounded up to 256 bytes, plus m doubles (256-
 * byte rounded) when chunk_scores is NULL and k int32 when sel_idx is NULL;
 * a shape needing more is refused with CKV_EINVAL before anything is
 * enqueued (the 32K-token 7B-shaped layer needs ~32 MB).  Every call on a
 * device uses that device's one array: calls that overlap in time on one
 * device (several streams or threads) race and must be serialized by the
 * caller.
 *   q, k_prefix, v_prefix, k_suffix, v_suffix, out: as ckv_reprefill_layer
 *   chunk_scores  device double[m] (written), or NULL
 *   sel_idx       device int32[k] (written, ascending), or NULL
 * k = ckv_num_keep(ceil(n/c), keep_ratio); asynchronous on `stream`.
 * ------------------------------------------------------------------------- */
#define CKV_NOALLOC_SCRATCH_BYTES (64u << 20)
ckv_status ckv_reprefill_layer_noalloc(const ckv_dims* dims, double keep_ratio, const void* q,
                                       const void* k_prefix, const void* v_prefix,
                                       const void* k_suffix, const void* v_suffix, void* out,
                                       double* chunk_scores, int32_t* sel_idx, void* stream);

/* ---------------------------------------------------------------------------
 * Read accounting -- Sec. 4.2 (a ContiguousChunk store reads exactly the
 * selected chunks) against Sec. 3, Motivation 1 (a store of fixed coarse
 * blocks reads every block that holds a needed token: read amplification).
 * For the selected chunks sel_idx[0..k) of an n-token prefix cut into chunks
 * of c tokens, counts what both stores read:
 *   tokens_selected  tokens of the selected chunks (the last chunk clamped to
 *                    n): what the ContiguousChunk store reads
 *   runs             maximal runs of consecutive selected chunks: contiguous
 *                    reads when adjacent chunks are merged
 *   blocks           blocks of block_tokens consecutive tokens (the
 *                    comparison systems use 64) holding a selected token
 *   tokens_block     tokens in those blocks (the last block clamped to n):
 *                    what the block store reads
 * Bytes are tokens times the bytes of one token's K and V in one layer; the
 * block store's read amplification is tokens_block / tokens_selected.
 *   sel_idx  host int32[k], strictly ascending, each in [0, ceil(n/c))
 *   k        0 <= k <= ceil(n/c)
 *   out      host, written
 * Host-only, pure, O(k).  CKV_EINVAL on n < 1, c < 1, block_tokens < 1, a
 * NULL pointer, or an index out of range or order (nothing written).
 * ------------------------------------------------------------------------- */
typedef struct ckv_io_counts {
  int64_t tokens_selected;
  int64_t runs;
  int64_t blocks;
  int64_t tokens_block;
} ckv_io_counts;
ckv_status ckv_io_account(int64_t n, int32_t c, const int32_t* sel_idx, int64_t k,
                          int32_t block_tokens, ckv_io_counts* out);

/* ---------------------------------------------------------------------------
 * Storage tier -- the prefix KV kept on SSD and loaded by I/O threads
 * (Sec. 4.3.2's loading steps; Sec. 4.5, where chunks missing from both
 * caches are loaded from SSD by I/O threads).
 * A store is one file of n_keys spans of span_bytes bytes; span `key` starts
 * at byte key * span_bytes.  For a layer context, key = layer * m + chunk and
 * a span is one chunk's K rows then V rows, c rows each (the host-resident
 * layout of ckv_layer_io.kv_host, layer after layer).  io_threads threads
 * (1..64) read; runs of consecutive keys going to consecutive destinations
 * are read with one pread, in pieces of at most 4 MiB.  CKV_STORE_DIRECT
 * opens the file with O_DIRECT (reads bypass the page cache), which needs
 * span_bytes to be a multiple of 4096; each I/O thread then reads into a
 * 4 MiB aligned buffer of its own and copies to the destination, so any
 * destination (pinned staging included) works.  CKV_EINVAL if the
 * file cannot be opened or is shorter than n_keys spans.  Host code; the file
 * is only read.
 * ------------------------------------------------------------------------- */
#define CKV_STORE_DIRECT 0x1
ckv_status ckv_store_open(const char* path, int64_t n_keys, int64_t span_bytes, int32_t io_threads,
                          int32_t flags, ckv_store** out);
/* Waits for the I/O threads to finish their queued reads, then closes. */
ckv_status ckv_store_close(ckv_store* store);
/* Reads spans keys[0..count) into dst (host memory, count consecutive spans)
 * with the I/O threads; returns when all have landed.  CKV_EINVAL on a key out
 * of range (nothing read), CKV_EHIP on a read error. */
ckv_status ckv_store_read(ckv_store* store, const int64_t* keys, int64_t count, void* dst);

/* ---------------------------------------------------------------------------
 * Attention-guided cache management -- Sec. 4.5, Eq. 2.
 * Decides which ContiguousChunks stay in GPU memory and in CPU memory across
 * requests.  Keys 0..n_keys-1 name cacheable chunks (for example
 * layer * m + chunk).  Each key keeps, for as long as the cache lives and
 * also after eviction (the in-memory score table):
 *   I  cumulative importance: the sum of the attention scores A_j (Eq. 1) of
 *      the requests that used the chunk,
 *   F  access frequency: the number of requests that used it, or, with
 *      CKV_CACHE_LOADS (the paper's wording read literally), the number of
 *      times it was loaded into GPU or CPU memory: its uses that found it
 *      outside the GPU tier,
 *   S  cache score I * F (CKV_CACHE_ATTENTION, CKV_CACHE_LOADS), or F alone
 *      (CKV_CACHE_LFU, the frequency-only policy of the ablation).
 * Two tiers of gpu_slots and cpu_slots entries are kept as min-heaps on
 * (S, time of latest access): the weakest entry is the one with the lowest S,
 * and among equal S the one accessed longest ago.
 * ckv_cache_access takes one request's used chunks in the given order; for
 * each it reports where the chunk was found (CKV_TIER_GPU: no transfer;
 * CKV_TIER_CPU: a CPU-to-GPU transfer; CKV_TIER_NONE: a load from storage),
 * adds A to I and one to F, and re-places it: into the GPU tier if there is
 * room or it outranks the GPU tier's weakest entry, which then moves to the
 * CPU tier by the same rule; otherwise into the CPU tier by that rule.  What
 * the CPU tier does not take leaves memory.  (The paper fixes the score, the
 * two heaps, the GPU-to-CPU cascade and the table; F counting requests, the
 * admission rule and the tie order are this library's reading.)  As S only
 * grows with each access, the GPU tier always holds the gpu_slots
 * highest-ranked chunks seen so far and the CPU tier the next cpu_slots.
 * The cache is host memory only and moves no data: the caller moves chunks
 * as the reported tiers say.  Not thread-safe; one cache per thread.
 * ------------------------------------------------------------------------- */
/* (ckv_cache is declared beside ckv_ctx above) */
#define CKV_CACHE_ATTENTION 0
#define CKV_CACHE_LFU 1
#define CKV_CACHE_LOADS 2
#define CKV_TIER_NONE 0
#define CKV_TIER_CPU 1
#define CKV_TIER_GPU 2

typedef struct ckv_cache_counts {
  int64_t hits_gpu; /* accessed chunks found in the GPU tier                 */
  int64_t hits_cpu; /* found in the CPU tier                                 */
  int64_t misses;   /* found in neither (loaded from storage)                */
  int64_t demoted;  /* GPU-tier evictions taken by the CPU tier              */
  int64_t dropped;  /* chunks that left memory or were not kept after a load */
} ckv_cache_counts;

/* n_keys >= 1, gpu_slots >= 0, cpu_slots >= 0, policy CKV_CACHE_ATTENTION,
 * CKV_CACHE_LFU or CKV_CACHE_LOADS.  Host allocation of O(n_keys + slots); CKV_ENOMEM on failure. */
ckv_status ckv_cache_create(int64_t n_keys, int64_t gpu_slots, int64_t cpu_slots, int32_t policy,
                            ckv_cache** out);
ckv_status ckv_cache_destroy(ckv_cache* cache);
/* One request: keys[count] distinct and in [0, n_keys), scores[count] finite
 * and >= 0 (the chunks' A_j).  tier_before[count] (may be NULL) receives the
 * tier each key was found in at its turn; *counts (may be NULL) the totals
 * since creation.  Everything is validated first: CKV_EINVAL changes nothing.
 * O(count * log(slots)). */
ckv_status ckv_cache_access(ckv_cache* cache, const int64_t* keys, const double* scores,
                            int64_t count, int8_t* tier_before, ckv_cache_counts* counts);
/* Current tier of keys[count] into tier[count]; changes nothing. */
ckv_status ckv_cache_lookup(const ckv_cache* cache, const int64_t* keys, int64_t count,
                            int8_t* tier);
/* I, F and tier of every key into arrays of n_keys entries (each may be NULL). */
ckv_status ckv_cache_state(const ckv_cache* cache, double* importance, int64_t* frequency,
                           int8_t* tier);
/* The keys of tier (CKV_TIER_CPU or CKV_TIER_GPU) in ascending order into
 * keys[0..capacity); *n receives the tier's size (CKV_EINVAL, nothing
 * written, if it exceeds capacity). */
ckv_status ckv_cache_resident(const ckv_cache* cache, int32_t tier, int64_t* keys,
                              int64_t capacity, int64_t* n);

#ifdef __cplusplus
}
#endif
#endif /* CKV_H */
