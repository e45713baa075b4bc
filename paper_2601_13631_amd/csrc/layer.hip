// layer.hip -- the Re-Prefill layer step and its context (ckv_ctx).
//
// HBM-resident prefix: score -> select -> attention reading the kept chunks'
// spans in place (or, with CKV_CTX_MATERIALIZE, gather -> attention over the
// compact copy), all on the caller's stream with no host synchronisation.
//
// Periods (Def. 4.2): with a Period of p layers (ckv_ctx_set_period), layer l
// runs scoring and selection only when l is a multiple of p; the other layers
// of the Period attend over the set that layer selected (kept in the context,
// on the device and, for a host-resident prefix, on the host), with no
// scoring, no selection and no host synchronisation.
//
// Host-resident prefix (Sec. 4.3.2): the K/V store
// of every layer lives in pinned host memory, chunk-major (chunk j of a layer
// is one span: K rows then V rows).  Two HBM slot buffers alternate between
// layers.  While layer l computes, the chunks that layer l selected are copied
// for layer l+1 into the other buffer on a prefetch stream (the prediction
// P_{l+1} = S_l).  When layer l+1 has selected S_{l+1}, only the difference
// S_{l+1} \ P_{l+1} is fetched on a demand stream into the free slots behind
// the prefetched ones, and the attention reads every kept chunk through a
// chunk -> slot table.  Copies move whole chunk spans, by a kernel that reads
// the pinned store over the host link (one launch per list of chunks instead
// of one DMA copy per run of consecutive chunks).  The selection is the
// step's only device -> host dependency.

#include <cstring>
#include <new>
#include <vector>

#include "tiers_internal.h"

using namespace ckv;

struct ckv_ctx {
  ckv_dims dims;
  double keep_ratio;
  int32_t flags;
  int64_t m, k;
  int device;
  // workspace (device)
  void* ws = nullptr;
  size_t ws_score = 0, ws_attn = 0, off_attn = 0, off_scores = 0, off_sel = 0, off_ksel = 0,
         off_vsel = 0, ws_bytes = 0;
  // host-resident prefix
  int64_t slot_bytes = 0;  // one chunk: K span + V span
  int64_t slots_per_buf = 0;
  // one arena of chunk slots: two transient buffers of slots_per_buf slots
  // (slots[0], slots[1]) then cache_slots slots holding the chunks of an
  // attached cache's GPU tier; slot tables index the whole arena
  void* arena = nullptr;
  void* slots[2] = {nullptr, nullptr};
  int32_t* slot_tab_dev[2] = {nullptr, nullptr};
  int32_t* sel_host = nullptr;      // pinned [k]
  int32_t* slot_tab_host[2] = {nullptr, nullptr};  // pinned [k]
  // chunk lists of the copy kernels: misses (demand) and the prediction
  // (prefetch) of each slot buffer, staged in pinned memory, read on the device
  int32_t* dem_host[2] = {nullptr, nullptr};
  int32_t* pref_host[2] = {nullptr, nullptr};
  int32_t* dem_dev[2] = {nullptr, nullptr};
  int32_t* pref_dev[2] = {nullptr, nullptr};
  hipStream_t demand = nullptr, prefetch = nullptr;
  hipEvent_t ev_sel = nullptr, ev_dem = nullptr, ev_pref[2] = {nullptr, nullptr},
             ev_attn[2] = {nullptr, nullptr};
  bool pref_pending[2] = {false, false}, attn_recorded[2] = {false, false};
  std::vector<int32_t> pred;  // prediction for the next layer (ascending), in slots 0..|pred|-1
  int32_t next_layer = 0;
  // Periods: layers period_first .. period_first+period-1 attend over the set
  // selected at period_first (device copy at off_pset, host copy pset_host)
  int32_t period = 1;
  int32_t period_first = -1;  // -1: no set held
  size_t off_pset = 0;
  std::vector<int32_t> pset_host;
  std::vector<double> pset_A;  // the Period set's chunk scores (attached cache only)
  // attention-guided cache (Sec. 4.5) attached to a host-resident prefix
  ckv_cache* cache = nullptr;
  int64_t cache_slots = 0, cache_layers = 0;
  std::vector<int32_t> slot_of;     // key -> cache slot, -1 if the chunk is not in HBM
  std::vector<int32_t> free_slots;  // cache slots holding nothing
  std::vector<int64_t> keys, evicted;
  std::vector<double> key_scores;
  double* scores_host = nullptr;                    // pinned [m]
  int32_t* fill_host[2] = {nullptr, nullptr};       // pinned [2k]: source slots, then target slots
  int32_t* fill_dev[2] = {nullptr, nullptr};
  bool pref_recorded[2] = {false, false};
  // storage tier: chunks come from a file into a pinned chunk pool, then to
  // HBM.  A chunk in an attached cache's GPU or CPU tier keeps its pool slot
  // (the pool is the CPU tier of Sec. 4.5, inclusive of the GPU tier); every
  // other slot is released, and reused only after the next layer's host
  // synchronisation, when the copies that read it have finished.
  ckv_store* kv_store = nullptr;
  int64_t store_layers = 0;
  char* pool = nullptr;  // pinned, pool_n slots of slot_bytes
  const void* pool_dev = nullptr;
  int64_t pool_n = 0;
  std::vector<int32_t> pool_of;  // key -> pool slot, -1 if its bytes are not in the pool
  std::vector<int32_t> pool_free, pool_quarantine;
  // copy lists (pool slots, then arena slots) of each buffer's prediction and
  // demand copies: pinned staging and device copies, 2 * slots_per_buf entries
  int32_t* xfer_host[2][2] = {{nullptr, nullptr}, {nullptr, nullptr}};
  int32_t* xfer_dev[2][2] = {{nullptr, nullptr}, {nullptr, nullptr}};
  // predictions read ahead from the store: entry layer % kAhead holds the
  // chunks (in P order) and keys read for that layer and the reads' ticket.
  // One layer ahead, or with a SubPeriod of sp layers inside a Period, up to
  // sp - 1 layers ahead (Sec. 4.3.2's intra-period prefetch).
  static constexpr int kAhead = 16;
  struct Ahead {
    int32_t layer = -1;
    int64_t ticket = 0;
    std::vector<int32_t> chunks;
    std::vector<int64_t> keys;
  };
  Ahead ahead[kAhead];
  int32_t subperiod = 1;
  std::vector<int64_t> io_keys, dropped;
  std::vector<char*> io_dst;
  std::vector<int32_t> xsrc, xdst;
  // stage timing: a ring of event sets, harvested when a set is reused or on query
  static constexpr int kRing = 64;
  hipEvent_t tev[kRing][CKV_N_STAGES + 1] = {};
  int64_t t_issued = 0, t_done = 0;
  double t_ms[CKV_N_STAGES] = {};
};

namespace {

// Waits for store reads into the pool that are still in flight.
void drain_store_reads(ckv_ctx* c) {
  for (auto& a : c->ahead) {
    if (c->kv_store && a.ticket) (void)store_wait(c->kv_store, a.ticket);
    a.ticket = 0;
  }
}

void free_pool(ckv_ctx* c) {
  (void)hipHostFree(c->pool);
  c->pool = nullptr;
  c->pool_dev = nullptr;
  c->pool_n = 0;
  for (int b = 0; b < 2; ++b)
    for (int i = 0; i < 2; ++i) {
      (void)hipHostFree(c->xfer_host[b][i]);
      (void)hipFree(c->xfer_dev[b][i]);
      c->xfer_host[b][i] = nullptr;
      c->xfer_dev[b][i] = nullptr;
    }
  c->pool_of.clear();
  c->pool_free.clear();
  c->pool_quarantine.clear();
  for (auto& a : c->ahead) {
    a.layer = -1;
    a.chunks.clear();
    a.keys.clear();
  }
}

// A free pool slot for the bytes of `key` (-1 if none is left).
int32_t pool_take(ckv_ctx* c, int64_t key) {
  if (c->pool_free.empty()) return -1;
  const int32_t sl = c->pool_free.back();
  c->pool_free.pop_back();
  c->pool_of[key] = sl;
  return sl;
}

// Releases key's pool slot; it becomes free after the next host synchronisation.
void pool_release(ckv_ctx* c, int64_t key) {
  if (c->pool_of[key] < 0) return;
  c->pool_quarantine.push_back(c->pool_of[key]);
  c->pool_of[key] = -1;
}

// Copies count chunks from pool slots src[] to arena slots dst[] on stream st,
// with the lists staged through this buffer's pinned and device arrays.
ckv_status pool_copy(ckv_ctx* c, int b, int which, const int32_t* src, const int32_t* dst,
                     int64_t count, hipStream_t st) {
  if (count == 0) return CKV_OK;
  const int64_t spb = c->slots_per_buf;
  int32_t* h = c->xfer_host[b][which];
  std::memcpy(h, src, (size_t)count * sizeof(int32_t));
  std::memcpy(h + spb, dst, (size_t)count * sizeof(int32_t));
  CKV_HIP(hipMemcpyAsync(c->xfer_dev[b][which], h, (size_t)(2 * spb) * sizeof(int32_t),
                         hipMemcpyHostToDevice, st));
  return launch_copy_slots(c->pool_dev, c->xfer_dev[b][which], c->arena,
                           c->xfer_dev[b][which] + spb, count, c->slot_bytes, st);
}

ckv_status free_ctx(ckv_ctx* c) {
  if (!c) return CKV_OK;
  drain_store_reads(c);
  if (c->cache) cache_log_gpu_evictions(c->cache, false);  // the cache outlives the context
  if (c->demand) (void)hipStreamSynchronize(c->demand);
  if (c->prefetch) (void)hipStreamSynchronize(c->prefetch);
  (void)hipFree(c->ws);
  for (int i = 0; i < 2; ++i) {
    (void)hipFree(c->slot_tab_dev[i]);
    (void)hipFree(c->fill_dev[i]);
    (void)hipHostFree(c->fill_host[i]);
    (void)hipHostFree(c->slot_tab_host[i]);
    (void)hipFree(c->dem_dev[i]);
    (void)hipFree(c->pref_dev[i]);
    (void)hipHostFree(c->dem_host[i]);
    (void)hipHostFree(c->pref_host[i]);
    if (c->ev_pref[i]) (void)hipEventDestroy(c->ev_pref[i]);
    if (c->ev_attn[i]) (void)hipEventDestroy(c->ev_attn[i]);
  }
  (void)hipFree(c->arena);
  free_pool(c);
  (void)hipHostFree(c->sel_host);
  (void)hipHostFree(c->scores_host);
  for (auto& set : c->tev)
    for (auto& e : set)
      if (e) (void)hipEventDestroy(e);
  if (c->ev_sel) (void)hipEventDestroy(c->ev_sel);
  if (c->ev_dem) (void)hipEventDestroy(c->ev_dem);
  if (c->demand) (void)hipStreamDestroy(c->demand);
  if (c->prefetch) (void)hipStreamDestroy(c->prefetch);
  delete c;
  return CKV_OK;
}

#define CKV_HIP_ALLOC(call)                                                              \
  do {                                                                                   \
    hipError_t e_ = (call);                                                              \
    if (e_ != hipSuccess) {                                                              \
      set_error("%s failed: %s", #call, hipGetErrorString(e_));                          \
      free_ctx(c);                                                                       \
      return e_ == hipErrorOutOfMemory ? CKV_ENOMEM : CKV_EHIP;                          \
    }                                                                                    \
  } while (0)

bool all_stages(const ckv_ctx* c) { return c->flags & CKV_CTX_STAGE_TIMING; }

// Adds the stage times of the oldest unaccounted layer to the totals.
ckv_status harvest_one(ckv_ctx* c) {
  hipEvent_t* e = c->tev[c->t_done % ckv_ctx::kRing];
  const int n = all_stages(c) ? CKV_N_STAGES : 1;
  CKV_HIP(hipEventSynchronize(e[n]));
  for (int s = 0; s < n; ++s) {
    float ms = 0.f;
    CKV_HIP(hipEventElapsedTime(&ms, e[s], e[s + 1]));
    c->t_ms[s] += ms;
  }
  ++c->t_done;
  return CKV_OK;
}

int64_t chunk_len(const ckv_dims* d, int64_t j) {
  return std::min<int64_t>(d->chunk_size, d->n_prefix - j * d->chunk_size);
}

}  // namespace

extern "C" {

ckv_status ckv_ctx_create(const ckv_dims* dims, double keep_ratio, int32_t flags, ckv_ctx** out) {
  clear_error();
  if (!out) CKV_FAIL(CKV_EINVAL, "out is NULL");
  *out = nullptr;
  {
    ckv_status s = check_dims(dims);
    if (s != CKV_OK) return s;
  }
  if (!(keep_ratio > 0.0 && keep_ratio <= 1.0)) CKV_FAIL(CKV_EINVAL, "keep_ratio must be in (0, 1]");
  if (flags & ~(CKV_CTX_HOST_PREFIX | CKV_CTX_MATERIALIZE | CKV_CTX_STAGE_TIMING |
                CKV_CTX_SCORE_TIMING))
    CKV_FAIL(CKV_EINVAL, "unknown flags");
  ckv_ctx* c = new (std::nothrow) ckv_ctx();
  if (!c) CKV_FAIL(CKV_ENOMEM, "host allocation failed");
  c->dims = *dims;
  c->keep_ratio = keep_ratio;
  c->flags = flags;
  c->m = ckv_num_chunks(dims->n_prefix, dims->chunk_size);
  c->k = ckv_num_keep(c->m, keep_ratio);
  CKV_HIP_ALLOC(hipGetDevice(&c->device));

  const int eb = elem_bytes(dims->dtype);
  const int64_t span = (int64_t)dims->chunk_size * dims->n_kv_heads * dims->head_dim * eb;
  c->ws_score = make_score_plan(dims).bytes;
  if (c->ws_score == 0) {
    free_ctx(c);
    CKV_FAIL(CKV_EUNSUPPORTED, "shape too large for the scoring decomposition");
  }
  c->ws_attn = make_attn_plan(dims, c->k).bytes;
  // scoring and attention scratch are used one after the other on one stream,
  // so both start at the front of the workspace
  c->off_attn = 0;
  size_t off = align_up(std::max(c->ws_score, c->ws_attn), 256);
  c->off_scores = off;
  off = align_up(off + (size_t)c->m * sizeof(double), 256);
  c->off_sel = off;
  off = align_up(off + (size_t)c->k * sizeof(int32_t), 256);
  c->off_pset = off;
  off = align_up(off + (size_t)c->k * sizeof(int32_t), 256);
  if (flags & CKV_CTX_MATERIALIZE) {
    c->off_ksel = off;
    off = align_up(off + (size_t)(c->k * span), 256);
    c->off_vsel = off;
    off = align_up(off + (size_t)(c->k * span), 256);
  }
  c->ws_bytes = off;
  CKV_HIP_ALLOC(hipMalloc(&c->ws, c->ws_bytes));

  if (flags & CKV_CTX_HOST_PREFIX) {
    c->slot_bytes = 2 * span;
    c->slots_per_buf = 2 * c->k;  // prefetched chunks plus room for a full miss set
    CKV_HIP_ALLOC(hipMalloc(&c->arena, (size_t)(2 * c->slots_per_buf * c->slot_bytes)));
    for (int i = 0; i < 2; ++i) {
      c->slots[i] = static_cast<char*>(c->arena) + i * c->slots_per_buf * c->slot_bytes;
      CKV_HIP_ALLOC(hipMalloc((void**)&c->fill_dev[i], (size_t)(2 * c->k) * sizeof(int32_t)));
      CKV_HIP_ALLOC(hipHostMalloc((void**)&c->fill_host[i], (size_t)(2 * c->k) * sizeof(int32_t),
                                  hipHostMallocDefault));
      CKV_HIP_ALLOC(hipMalloc((void**)&c->slot_tab_dev[i], (size_t)c->k * sizeof(int32_t)));
      CKV_HIP_ALLOC(hipHostMalloc((void**)&c->slot_tab_host[i], (size_t)c->k * sizeof(int32_t),
                                  hipHostMallocDefault));
      CKV_HIP_ALLOC(hipMalloc((void**)&c->dem_dev[i], (size_t)c->k * sizeof(int32_t)));
      CKV_HIP_ALLOC(hipMalloc((void**)&c->pref_dev[i], (size_t)c->k * sizeof(int32_t)));
      CKV_HIP_ALLOC(hipHostMalloc((void**)&c->dem_host[i], (size_t)c->k * sizeof(int32_t),
                                  hipHostMallocDefault));
      CKV_HIP_ALLOC(hipHostMalloc((void**)&c->pref_host[i], (size_t)c->k * sizeof(int32_t),
                                  hipHostMallocDefault));
      CKV_HIP_ALLOC(hipEventCreateWithFlags(&c->ev_pref[i], hipEventDisableTiming));
      CKV_HIP_ALLOC(hipEventCreateWithFlags(&c->ev_attn[i], hipEventDisableTiming));
    }
    CKV_HIP_ALLOC(hipHostMalloc((void**)&c->sel_host, (size_t)c->k * sizeof(int32_t),
                                hipHostMallocDefault));
    CKV_HIP_ALLOC(hipHostMalloc((void**)&c->scores_host, (size_t)c->m * sizeof(double),
                                hipHostMallocDefault));
    CKV_HIP_ALLOC(hipStreamCreateWithFlags(&c->demand, hipStreamNonBlocking));
    CKV_HIP_ALLOC(hipStreamCreateWithFlags(&c->prefetch, hipStreamNonBlocking));
    CKV_HIP_ALLOC(hipEventCreateWithFlags(&c->ev_sel, hipEventDisableTiming));
    CKV_HIP_ALLOC(hipEventCreateWithFlags(&c->ev_dem, hipEventDisableTiming));
  }
  if (flags & (CKV_CTX_STAGE_TIMING | CKV_CTX_SCORE_TIMING))
    for (auto& set : c->tev)
      for (auto& e : set) CKV_HIP_ALLOC(hipEventCreate(&e));
  *out = c;
  return CKV_OK;
}

ckv_status ckv_ctx_stage_times(ckv_ctx* ctx, double* ms, int64_t* n_layers) {
  clear_error();
  if (!ctx || !ms || !n_layers) CKV_FAIL(CKV_EINVAL, "NULL argument");
  if (!(ctx->flags & (CKV_CTX_STAGE_TIMING | CKV_CTX_SCORE_TIMING)))
    CKV_FAIL(CKV_ESTATE, "context created without CKV_CTX_STAGE_TIMING or CKV_CTX_SCORE_TIMING");
  while (ctx->t_done < ctx->t_issued) {
    ckv_status s = harvest_one(ctx);
    if (s != CKV_OK) return s;
  }
  for (int s = 0; s < CKV_N_STAGES; ++s) ms[s] = ctx->t_ms[s];
  *n_layers = ctx->t_done;
  return CKV_OK;
}

ckv_status ckv_ctx_destroy(ckv_ctx* ctx) { return free_ctx(ctx); }

ckv_status ckv_ctx_set_period(ckv_ctx* ctx, int32_t period) {
  clear_error();
  if (!ctx) CKV_FAIL(CKV_EINVAL, "ctx is NULL");
  if (period < 1) CKV_FAIL(CKV_EINVAL, "period must be >= 1 (got %d)", period);
  ctx->period = period;
  ctx->period_first = -1;
  return CKV_OK;
}

ckv_status ckv_ctx_attach_cache(ckv_ctx* ctx, ckv_cache* cache) {
  clear_error();
  if (!ctx) CKV_FAIL(CKV_EINVAL, "ctx is NULL");
  if (!(ctx->flags & CKV_CTX_HOST_PREFIX))
    CKV_FAIL(CKV_EINVAL, "a cache needs a context with a host-resident prefix");
  if (ctx->next_layer != 0)
    CKV_FAIL(CKV_ESTATE, "attach a cache at the start of a request (before layer 0 or after a reset)");
  if (ctx->kv_store)
    CKV_FAIL(CKV_ESTATE, "attach the cache before the store (the store's chunk pool holds its tiers)");
  int64_t G = 0;
  if (cache) {
    if (cache_keys(cache) % ctx->m != 0)
      CKV_FAIL(CKV_EINVAL, "cache keys (%lld) must be a whole number of layers of %lld chunks",
               (long long)cache_keys(cache), (long long)ctx->m);
    if (cache_gpu_size(cache) != 0)
      CKV_FAIL(CKV_ESTATE, "the cache's GPU tier must be empty when it is attached");
    G = std::min(cache_gpu_slots(cache), cache_keys(cache));
    if (2 * ctx->slots_per_buf + G > INT32_MAX)
      CKV_FAIL(CKV_EUNSUPPORTED, "too many cache slots (%lld)", (long long)G);
  }
  // the arena is replaced with nothing in flight that could still read it
  CKV_HIP(hipDeviceSynchronize());
  const size_t bytes = (size_t)((2 * ctx->slots_per_buf + G) * ctx->slot_bytes);
  void* arena = nullptr;
  hipError_t e = hipMalloc(&arena, bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    CKV_FAIL(e == hipErrorOutOfMemory ? CKV_ENOMEM : CKV_EHIP, "hipMalloc of %zu bytes of cache slots failed: %s",
             bytes, hipGetErrorString(e));
  }
  CKV_HIP(hipFree(ctx->arena));
  ctx->arena = arena;
  for (int i = 0; i < 2; ++i)
    ctx->slots[i] = static_cast<char*>(arena) + i * ctx->slots_per_buf * ctx->slot_bytes;
  if (ctx->cache) cache_log_gpu_evictions(ctx->cache, false);
  ctx->cache = cache;
  ctx->cache_slots = G;
  ctx->cache_layers = cache ? cache_keys(cache) / ctx->m : 0;
  ctx->slot_of.assign(cache ? (size_t)cache_keys(cache) : 0, -1);
  ctx->free_slots.clear();
  for (int64_t i = G - 1; i >= 0; --i) ctx->free_slots.push_back((int32_t)i);
  if (cache) cache_log_gpu_evictions(cache, true);
  return CKV_OK;
}

ckv_status ckv_ctx_set_subperiod(ckv_ctx* ctx, int32_t subperiod) {
  clear_error();
  if (!ctx) CKV_FAIL(CKV_EINVAL, "ctx is NULL");
  if (subperiod < 1 || subperiod > ckv_ctx::kAhead)
    CKV_FAIL(CKV_EINVAL, "subperiod must be in [1, %d] (got %d)", ckv_ctx::kAhead, subperiod);
  if (ctx->kv_store)
    CKV_FAIL(CKV_ESTATE, "set the SubPeriod before attaching the store (it sizes the chunk pool)");
  ctx->subperiod = subperiod;
  return CKV_OK;
}

ckv_status ckv_ctx_attach_store(ckv_ctx* ctx, ckv_store* store) {
  clear_error();
  if (!ctx) CKV_FAIL(CKV_EINVAL, "ctx is NULL");
  if (!(ctx->flags & CKV_CTX_HOST_PREFIX))
    CKV_FAIL(CKV_EINVAL, "a store needs a context with a host-resident prefix");
  if (ctx->next_layer != 0)
    CKV_FAIL(CKV_ESTATE, "attach a store at the start of a request (before layer 0 or after a reset)");
  if (store) {
    if (store_span_bytes(store) != ctx->slot_bytes)
      CKV_FAIL(CKV_EINVAL, "store spans of %lld bytes, chunks of %lld", (long long)store_span_bytes(store),
               (long long)ctx->slot_bytes);
    if (store_keys(store) % ctx->m != 0)
      CKV_FAIL(CKV_EINVAL, "store keys (%lld) must be a whole number of layers of %lld chunks",
               (long long)store_keys(store), (long long)ctx->m);
    if (ctx->cache && cache_keys(ctx->cache) != store_keys(store))
      CKV_FAIL(CKV_EINVAL, "the attached cache and the store name different key ranges");
  }
  drain_store_reads(ctx);
  CKV_HIP(hipDeviceSynchronize());
  free_pool(ctx);
  ctx->kv_store = nullptr;
  ctx->store_layers = 0;
  if (!store) return CKV_OK;
  // room for the cache's tiers, plus the transient chunks of two layers in
  // flight and of the layer whose slots wait for release
  const int64_t keys = store_keys(store), k = ctx->k;
  const int64_t kept = ctx->cache ? std::min(keys, cache_gpu_slots(ctx->cache) + cache_cpu_slots(ctx->cache)) : 0;
  const int64_t n = std::min(keys, kept + (6 + ctx->subperiod) * k) + 16;
  const int64_t spb = ctx->slots_per_buf;
  hipError_t e = hipHostMalloc((void**)&ctx->pool, (size_t)(n * ctx->slot_bytes), hipHostMallocDefault);
  for (int b = 0; b < 2 && e == hipSuccess; ++b)
    for (int i = 0; i < 2 && e == hipSuccess; ++i) {
      e = hipHostMalloc((void**)&ctx->xfer_host[b][i], (size_t)(2 * spb) * sizeof(int32_t),
                        hipHostMallocDefault);
      if (e == hipSuccess) e = hipMalloc((void**)&ctx->xfer_dev[b][i], (size_t)(2 * spb) * sizeof(int32_t));
    }
  if (e != hipSuccess) {
    free_pool(ctx);
    CKV_FAIL(e == hipErrorOutOfMemory ? CKV_ENOMEM : CKV_EHIP, "pinned chunk pool of %lld slots: %s",
             (long long)n, hipGetErrorString(e));
  }
  ctx->pool_dev = device_view(ctx->pool);
  if (!ctx->pool_dev) {
    free_pool(ctx);
    CKV_FAIL(CKV_EHIP, "the pinned chunk pool is not visible to the device");
  }
  ctx->pool_n = n;
  ctx->pool_of.assign((size_t)keys, -1);
  for (int64_t i = n - 1; i >= 0; --i) ctx->pool_free.push_back((int32_t)i);
  ctx->kv_store = store;
  ctx->store_layers = keys / ctx->m;
  return CKV_OK;
}

ckv_status ckv_ctx_reset(ckv_ctx* ctx) {
  clear_error();
  if (!ctx) CKV_FAIL(CKV_EINVAL, "ctx is NULL");
  if (ctx->prefetch) CKV_HIP(hipStreamSynchronize(ctx->prefetch));
  drain_store_reads(ctx);
  if (ctx->kv_store) {
    // predictions read for a layer that will not run: release their slots
    // (nothing reads them any more once the device is idle)
    CKV_HIP(hipDeviceSynchronize());
    for (auto& a : ctx->ahead) {
      for (int64_t x : a.keys)
        if (!ctx->cache || cache_tier(ctx->cache, x) == CKV_TIER_NONE) pool_release(ctx, x);
      a.layer = -1;
      a.chunks.clear();
      a.keys.clear();
    }
  }
  ctx->pred.clear();
  ctx->pref_pending[0] = ctx->pref_pending[1] = false;
  ctx->next_layer = 0;
  ctx->period_first = -1;
  while (ctx->t_done < ctx->t_issued) {
    ckv_status s = harvest_one(ctx);
    if (s != CKV_OK) return s;
  }
  for (double& x : ctx->t_ms) x = 0.0;
  ctx->t_done = ctx->t_issued = 0;
  return CKV_OK;
}

ckv_status ckv_reprefill_layer(ckv_ctx* c, int32_t layer, const ckv_layer_io* io,
                               ckv_layer_stats* stats) {
  clear_error();
  if (!c || !io) CKV_FAIL(CKV_EINVAL, "NULL ctx or io");
  const ckv_dims* d = &c->dims;
  const bool host = c->flags & CKV_CTX_HOST_PREFIX;
  const void* store = nullptr;       // kv_host as the device reads it
  const void* store_next = nullptr;  // kv_host_next as the device reads it
  if (!io->q || !io->k_suffix || !io->v_suffix || !io->k_probe || !io->out)
    CKV_FAIL(CKV_EINVAL, "NULL tensor in io");
  if (!aligned16(io->q) || !aligned16(io->k_suffix) || !aligned16(io->v_suffix) ||
      !aligned16(io->k_probe) || !aligned16(io->out))
    CKV_FAIL(CKV_EINVAL, "tensors must be 16-byte aligned");
  const bool stored = host && c->kv_store;  // chunks come from the storage tier
  if (stored) {
    if (layer != c->next_layer)
      CKV_FAIL(CKV_ESTATE, "host-resident layers must run in order (expected %d, got %d)",
               c->next_layer, layer);
    if (layer >= c->store_layers)
      CKV_FAIL(CKV_EINVAL, "layer %d is not in the attached store (%lld layers)", layer,
               (long long)c->store_layers);
  } else if (host) {
    if (!io->kv_host) CKV_FAIL(CKV_EINVAL, "host-resident prefix needs kv_host");
    if (layer != c->next_layer)
      CKV_FAIL(CKV_ESTATE, "host-resident layers must run in order (expected %d, got %d)",
               c->next_layer, layer);
    // the copy kernels read the stores through the device's mapping of them
    store = device_view(io->kv_host);
    if (!store) CKV_FAIL(CKV_EINVAL, "kv_host must be pinned host memory (hipHostMalloc)");
    if (io->kv_host_next) {
      store_next = device_view(io->kv_host_next);
      if (!store_next) CKV_FAIL(CKV_EINVAL, "kv_host_next must be pinned host memory (hipHostMalloc)");
    }
  } else {
    if (!io->k_prefix || !io->v_prefix) CKV_FAIL(CKV_EINVAL, "HBM-resident prefix needs k/v_prefix");
    if (!aligned16(io->k_prefix) || !aligned16(io->v_prefix))
      CKV_FAIL(CKV_EINVAL, "tensors must be 16-byte aligned");
  }
  if (layer < 0) CKV_FAIL(CKV_EINVAL, "layer must be >= 0 (got %d)", layer);
  if (host && c->cache && layer >= c->cache_layers)
    CKV_FAIL(CKV_EINVAL, "layer %d has no keys in the attached cache (%lld layers)", layer,
             (long long)c->cache_layers);
  // a layer past the first of its Period reuses the set selected there
  const int32_t first = layer - layer % c->period;
  const bool reuse = first != layer;
  if (reuse && c->period_first != first)
    CKV_FAIL(CKV_ESTATE, "layer %d reuses the set of layer %d, the first of its Period, which has not run",
             layer, first);
  hipStream_t st = (hipStream_t)io->stream;
  char* ws = static_cast<char*>(c->ws);
  double* scores = io->chunk_scores ? io->chunk_scores : reinterpret_cast<double*>(ws + c->off_scores);
  int32_t* pset = reinterpret_cast<int32_t*>(ws + c->off_pset);
  // the set this layer attends over: selected now, or the Period's
  int32_t* sel = reuse ? pset : io->sel_idx ? io->sel_idx : reinterpret_cast<int32_t*>(ws + c->off_sel);
  const int64_t k = c->k;
  const int eb = elem_bytes(d->dtype);
  const int64_t span_elems = (int64_t)d->chunk_size * d->n_kv_heads * d->head_dim;

  hipEvent_t* tev = nullptr;
  // a reused layer has no scoring kernel to time alone
  if ((c->flags & CKV_CTX_STAGE_TIMING) || ((c->flags & CKV_CTX_SCORE_TIMING) && !reuse)) {
    if (c->t_issued - c->t_done >= ckv_ctx::kRing) {  // reuse the oldest set: account it first
      ckv_status s = harvest_one(c);
      if (s != CKV_OK) return s;
    }
    tev = c->tev[c->t_issued % ckv_ctx::kRing];
    // every stage: the set starts here; the scoring kernel alone: its own
    // launch brackets it (bf16), else the set starts here too
    if (all_stages(c) || d->dtype != CKV_DTYPE_BF16) CKV_HIP(hipEventRecord(tev[0], st));
  }
  auto mark = [&](int i) -> ckv_status {
    if (tev && all_stages(c)) CKV_HIP(hipEventRecord(tev[i], st));
    return CKV_OK;
  };

  ckv_status s = CKV_OK;
  if (!reuse) {
    const bool bracket = tev && !all_stages(c) && d->dtype == CKV_DTYPE_BF16;
    s = launch_score(d, io->q, io->k_probe, scores, ws, c->ws_score, st, tev ? tev[1] : nullptr,
                     bracket ? tev[0] : nullptr);
    if (s != CKV_OK) return s;
    if ((s = mark(2)) != CKV_OK) return s;
    s = launch_select(scores, c->m, k, sel, nullptr, 0, st);
    if (s != CKV_OK) return s;
    if ((s = mark(3)) != CKV_OK) return s;
    if (c->period > 1) {  // keep the set for the rest of the Period
      CKV_HIP(hipMemcpyAsync(pset, sel, (size_t)k * sizeof(int32_t), hipMemcpyDeviceToDevice, st));
      c->period_first = layer;
    }
  } else {
    if ((s = mark(1)) != CKV_OK) return s;
    if ((s = mark(2)) != CKV_OK) return s;
    if (io->sel_idx)  // the caller sees the set the layer used
      CKV_HIP(hipMemcpyAsync(io->sel_idx, pset, (size_t)k * sizeof(int32_t),
                             hipMemcpyDeviceToDevice, st));
    if ((s = mark(3)) != CKV_OK) return s;
  }

  ckv_layer_stats stv{};
  stv.k = k;
  if (!host) {
    ChunkSource src{io->k_prefix, io->v_prefix, span_elems, nullptr, 1};
    if (c->flags & CKV_CTX_MATERIALIZE) {
      void* ksel = ws + c->off_ksel;
      void* vsel = ws + c->off_vsel;
      s = launch_gather(d, io->k_prefix, io->v_prefix, sel, k, ksel, vsel, st);
      if (s != CKV_OK) return s;
      src = ChunkSource{ksel, vsel, span_elems, nullptr, 0};
    }
    if ((s = mark(4)) != CKV_OK) return s;
    s = launch_attn(d, io->q, src, sel, k, io->k_suffix, io->v_suffix, io->out, ws + c->off_attn,
                    c->ws_attn, st);
    if (s != CKV_OK) return s;
    if ((s = mark(5)) != CKV_OK) return s;
    if (tev) ++c->t_issued;
    // K+V bytes of k full chunks (the set stays on the device, so a short last
    // chunk, if kept, is counted at full length)
    stv.bytes_gathered = 2 * k * span_elems * eb;
    if (stats) *stats = stv;
    return CKV_OK;
  }

  // ---- host-resident prefix ------------------------------------------------
  const int cur = layer & 1, nxt = cur ^ 1;
  const bool cached = c->cache != nullptr;
  const int64_t key0 = (int64_t)layer * c->m;
  const int64_t spb = c->slots_per_buf;
  const int64_t buf0 = cur * spb, cache0 = 2 * spb;
  ckv_ctx::Ahead& mine = c->ahead[layer % ckv_ctx::kAhead];
  if (stored) {  // this layer's prediction: read (or queued) during earlier layers
    if (mine.layer != layer) {
      mine.layer = -1;
      mine.chunks.clear();
      mine.keys.clear();
    }
    if (mine.ticket) {
      s = store_wait(c->kv_store, mine.ticket);
      mine.ticket = 0;
      if (s != CKV_OK) return s;
    }
    c->pred = mine.chunks;
  }
  if (stored && !mine.keys.empty()) {
    // the predicted chunks (read from the store, or already in the pool) move
    // to this layer's HBM slots 0..|P|-1 on the prefetch stream, beside this
    // layer's scoring; this buffer's copy lists were last read two layers ago
    const std::vector<int64_t>& pk = mine.keys;
    const int64_t np = (int64_t)pk.size();
    c->xsrc.resize((size_t)np);
    c->xdst.resize((size_t)np);
    for (int64_t i = 0; i < np; ++i) {
      c->xsrc[i] = c->pool_of[pk[i]];
      c->xdst[i] = (int32_t)(buf0 + i);
      if (c->xsrc[i] < 0) CKV_FAIL(CKV_ESTATE, "predicted chunk not in the pool (internal)");
    }
    if (c->attn_recorded[cur]) {
      CKV_HIP(hipEventSynchronize(c->ev_attn[cur]));
      CKV_HIP(hipStreamWaitEvent(c->prefetch, c->ev_attn[cur], 0));
    }
    CKV_HIP(hipStreamWaitEvent(c->prefetch, c->ev_dem, 0));
    s = pool_copy(c, cur, 0, c->xsrc.data(), c->xdst.data(), np, c->prefetch);
    if (s != CKV_OK) return s;
    CKV_HIP(hipEventRecord(c->ev_pref[cur], c->prefetch));
    c->pref_pending[cur] = true;
    c->pref_recorded[cur] = true;
  }
  if (reuse) {  // the Period's set is already on the host: no synchronisation
    if (cached || stored) {
      // the host staging written below was last read by the copies of two
      // layers ago (and the prefetch list, or the store's staging buffer, by
      // the previous layer's); their contents differ from layer to layer
      if (c->attn_recorded[cur]) CKV_HIP(hipEventSynchronize(c->ev_attn[cur]));
      if (c->pref_recorded[nxt]) CKV_HIP(hipEventSynchronize(c->ev_pref[nxt]));
      if (stored && c->attn_recorded[nxt]) CKV_HIP(hipEventSynchronize(c->ev_attn[nxt]));
    }
    std::memcpy(c->sel_host, c->pset_host.data(), (size_t)k * sizeof(int32_t));
  } else {
    CKV_HIP(hipMemcpyAsync(c->sel_host, sel, (size_t)k * sizeof(int32_t), hipMemcpyDeviceToHost, st));
    if (cached)
      CKV_HIP(hipMemcpyAsync(c->scores_host, scores, (size_t)c->m * sizeof(double),
                             hipMemcpyDeviceToHost, st));
    CKV_HIP(hipEventRecord(c->ev_sel, st));
    CKV_HIP(hipEventSynchronize(c->ev_sel));
    if (c->period > 1) {
      c->pset_host.assign(c->sel_host, c->sel_host + k);
      if (cached) {
        c->pset_A.resize((size_t)k);
        for (int64_t u = 0; u < k; ++u) c->pset_A[u] = c->scores_host[c->sel_host[u]];
      }
    }
  }
  if (stored) {  // the previous layer's copies have finished: its released slots are free
    c->pool_free.insert(c->pool_free.end(), c->pool_quarantine.begin(), c->pool_quarantine.end());
    c->pool_quarantine.clear();
  }

  // slot table, in arena slots: chunks held in the cache's HBM slots are read
  // there; predicted chunks sit in this layer's buffer at slots 0..|P|-1 (in P
  // order), misses follow
  const std::vector<int32_t>& P = c->pred;
  std::vector<int32_t> miss;
  miss.reserve((size_t)k);
  int32_t* tab = c->slot_tab_host[cur];
  size_t pi = 0;
  int64_t hits = 0;
  for (int64_t u = 0; u < k; ++u) {
    const int32_t j = c->sel_host[u];
    const int64_t chunk_bytes = 2 * chunk_len(d, j) * d->n_kv_heads * d->head_dim * eb;
    stv.bytes_gathered += chunk_bytes;
    if (cached && c->slot_of[key0 + j] >= 0) {
      tab[u] = (int32_t)(cache0 + c->slot_of[key0 + j]);
      ++stv.cache_hits;
      continue;
    }
    while (pi < P.size() && P[pi] < j) ++pi;
    if (pi < P.size() && P[pi] == j) {
      tab[u] = (int32_t)(buf0 + pi);
      ++hits;
    } else {
      tab[u] = (int32_t)(buf0 + P.size() + miss.size());
      miss.push_back(j);
      stv.bytes_demand += chunk_bytes;
    }
  }
  stv.hits = hits;
  stv.misses = (int64_t)miss.size();
  stv.wasted = (int64_t)P.size() - hits;
  // misses follow the predicted chunks in this layer's buffer (c->pred is
  // replaced by the next layer's prediction below)
  const int64_t n_pred = (int64_t)P.size();

  // storage tier: the pool slots the misses move from; those not in the pool
  // get free slots and are read from the file below
  c->io_keys.clear();  // this layer's demand reads (none without misses)
  c->io_dst.clear();
  if (stored && !miss.empty()) {
    const size_t nm = miss.size();
    c->xsrc.resize(nm);
    c->xdst.resize(nm);
    for (size_t i = 0; i < nm; ++i) {
      const int64_t x = key0 + miss[i];
      if (c->pool_of[x] < 0) {
        if (pool_take(c, x) < 0) CKV_FAIL(CKV_ESTATE, "chunk pool exhausted (internal)");
        c->io_keys.push_back(x);
        c->io_dst.push_back(c->pool + (int64_t)c->pool_of[x] * c->slot_bytes);
      }
      c->xsrc[i] = c->pool_of[x];
      c->xdst[i] = (int32_t)(buf0 + n_pred + i);
    }
  }
  // the storage tier's demand reads start now; the layer waits for them below
  int64_t dem_ticket = 0;
  if (!c->io_keys.empty()) {
    s = store_submit(c->kv_store, c->io_keys.data(), (int64_t)c->io_keys.size(), c->io_dst.data(),
                     &dem_ticket);
    if (s != CKV_OK) return s;
    stv.bytes_storage += (int64_t)c->io_keys.size() * c->slot_bytes;
  }

  // demand copies into this layer's buffer (after the attention that last used
  // it; from the pool once its reads have landed), then the attention.  The
  // small index copies go first, so they never queue behind span copies.
  auto demand_and_attention = [&]() -> ckv_status {
    if (dem_ticket) {
      ckv_status w = store_wait(c->kv_store, dem_ticket);
      if (w != CKV_OK) return w;
    }
    if (c->attn_recorded[cur]) CKV_HIP(hipStreamWaitEvent(c->demand, c->ev_attn[cur], 0));
    CKV_HIP(hipMemcpyAsync(c->slot_tab_dev[cur], tab, (size_t)k * sizeof(int32_t),
                           hipMemcpyHostToDevice, c->demand));
    ckv_status r = CKV_OK;
    if (!miss.empty() && stored) {
      r = pool_copy(c, cur, 1, c->xsrc.data(), c->xdst.data(), (int64_t)miss.size(), c->demand);
    } else if (!miss.empty()) {
      std::memcpy(c->dem_host[cur], miss.data(), miss.size() * sizeof(int32_t));
      CKV_HIP(hipMemcpyAsync(c->dem_dev[cur], c->dem_host[cur], miss.size() * sizeof(int32_t),
                             hipMemcpyHostToDevice, c->demand));
      r = launch_copy_spans(store, c->dem_dev[cur], (int64_t)miss.size(), n_pred, c->slots[cur],
                            c->slot_bytes, c->demand);
    }
    if (r != CKV_OK) return r;
    CKV_HIP(hipEventRecord(c->ev_dem, c->demand));
    CKV_HIP(hipStreamWaitEvent(st, c->ev_dem, 0));
    if (c->pref_pending[cur]) CKV_HIP(hipStreamWaitEvent(st, c->ev_pref[cur], 0));
    c->pref_pending[cur] = false;
    if ((r = mark(4)) != CKV_OK) return r;
    ChunkSource src{c->arena, static_cast<char*>(c->arena) + span_elems * eb, 2 * span_elems,
                    c->slot_tab_dev[cur], 0};
    r = launch_attn(d, io->q, src, sel, k, io->k_suffix, io->v_suffix, io->out, ws + c->off_attn,
                    c->ws_attn, st);
    if (r != CKV_OK) return r;
    if ((r = mark(5)) != CKV_OK) return r;
    if (tev) ++c->t_issued;
    return CKV_OK;
  };
  // from pinned host memory the attention goes out first and the host work
  // below overlaps it; from the store the host works while the reads land
  if (!stored && (s = demand_and_attention()) != CKV_OK) return s;

  // Sec. 4.5: the chunks this layer uses add their scores (I += A, F += 1) and
  // are re-placed.  Chunks leaving the GPU tier free their HBM slots, and
  // chunks entering it are listed for copies from this layer's buffer, which
  // go on the stream after the attention that reads both.
  int64_t nf = 0;
  if (cached) {
    c->keys.resize((size_t)k);
    c->key_scores.resize((size_t)k);
    for (int64_t u = 0; u < k; ++u) {
      c->keys[u] = key0 + c->sel_host[u];
      c->key_scores[u] = reuse ? c->pset_A[u] : c->scores_host[c->sel_host[u]];
    }
    s = ckv_cache_access(c->cache, c->keys.data(), c->key_scores.data(), k, nullptr, nullptr);
    if (s != CKV_OK) return s;
    cache_take_gpu_evictions(c->cache, c->evicted);
    // the keys sent out of memory (used by the storage tier's pool below; the
    // log is drained every layer either way)
    cache_take_drops(c->cache, c->dropped);
    // a chunk displaced by an earlier chunk of this layer and placed back at
    // its own turn is still in the GPU tier: it keeps its slot and its bytes
    for (int64_t x : c->evicted)
      if (c->slot_of[x] >= 0 && cache_tier(c->cache, x) != CKV_TIER_GPU) {
        c->free_slots.push_back(c->slot_of[x]);
        c->slot_of[x] = -1;
      }
    int32_t* fill = c->fill_host[cur];
    for (int64_t u = 0; u < k; ++u) {
      const int64_t x = c->keys[u];
      if (cache_tier(c->cache, x) != CKV_TIER_GPU || c->slot_of[x] >= 0) continue;
      if (c->free_slots.empty()) CKV_FAIL(CKV_ESTATE, "cache slots exhausted (internal)");
      c->slot_of[x] = c->free_slots.back();
      c->free_slots.pop_back();
      fill[nf] = tab[u];
      fill[k + nf] = (int32_t)(cache0 + c->slot_of[x]);
      ++nf;
    }
  }
  if (stored) {
    // the pool keeps the chunks the cache holds (GPU or CPU tier); this layer's
    // other chunks, its unused predicted chunks and the chunks the cascade sent
    // out of memory release their slots (reused only after the next layer's
    // host synchronisation, when this layer's copies out of them are done)
    auto keep = [&](int64_t x) { return cached && cache_tier(c->cache, x) != CKV_TIER_NONE; };
    if (cached)
      for (int64_t x : c->dropped)
        if (!keep(x)) pool_release(c, x);
    for (int64_t u = 0; u < k; ++u)
      if (!keep(key0 + c->sel_host[u])) pool_release(c, key0 + c->sel_host[u]);
    for (int64_t x : mine.keys)
      if (!keep(x)) pool_release(c, x);
    mine.layer = -1;
    mine.chunks.clear();
    mine.keys.clear();
  }

  // the next layer's prediction (P_{l+1} = S_l) less the chunks it will find in
  // the cache's HBM slots
  c->pred.clear();
  const bool has_next = stored ? layer + 1 < c->store_layers : io->kv_host_next != nullptr;
  const int64_t nkey0 = (int64_t)(layer + 1) * c->m;
  if (has_next) {
    const bool next_cached = cached && layer + 1 < c->cache_layers;
    for (int64_t u = 0; u < k; ++u) {
      const int32_t j = c->sel_host[u];
      if (next_cached && c->slot_of[nkey0 + j] >= 0) continue;
      c->pred.push_back(j);
    }
    if (!stored)  // the storage tier counts what it queues, below
      for (int32_t j : c->pred)
        stv.bytes_prefetch += 2 * chunk_len(d, j) * d->n_kv_heads * d->head_dim * eb;
  }
  const int64_t np = (int64_t)c->pred.size();

  if (stored) {
    // the next layer's prediction joins the I/O threads' queue behind this
    // layer's demand reads and runs on while this layer attends and the next
    // one scores
    if (has_next) {
      // layers last_ahead..: inside a Period with a SubPeriod of sp layers,
      // every layer up to sp - 1 ahead (their set is this one); otherwise the
      // next layer only (speculative across a Period boundary)
      int64_t last_ahead = layer + 1;
      if (c->period > 1 && c->subperiod > 1) {
        const int64_t period_end = first + c->period - 1;
        last_ahead = std::max<int64_t>(last_ahead, std::min<int64_t>(layer + c->subperiod - 1, period_end));
      }
      last_ahead = std::min<int64_t>(last_ahead, c->store_layers - 1);
      for (int64_t t = layer + 1; t <= last_ahead; ++t) {
        ckv_ctx::Ahead& a = c->ahead[t % ckv_ctx::kAhead];
        if (a.layer == t) continue;  // queued by an earlier layer of the Period
        if (a.layer >= 0) CKV_FAIL(CKV_ESTATE, "prediction ring overrun (internal)");
        a.layer = (int32_t)t;
        a.chunks.clear();
        a.keys.clear();
        c->io_keys.clear();
        c->io_dst.clear();
        const int64_t tkey0 = t * c->m;
        const bool t_cached = cached && t < c->cache_layers;
        for (int64_t u = 0; u < k; ++u) {
          const int32_t j = c->sel_host[u];
          const int64_t x = tkey0 + j;
          if (t_cached && c->slot_of[x] >= 0) continue;
          a.chunks.push_back(j);
          a.keys.push_back(x);
          stv.bytes_prefetch += 2 * chunk_len(d, j) * d->n_kv_heads * d->head_dim * eb;
          if (c->pool_of[x] >= 0) continue;
          if (pool_take(c, x) < 0) CKV_FAIL(CKV_ESTATE, "chunk pool exhausted (internal)");
          c->io_keys.push_back(x);
          c->io_dst.push_back(c->pool + (int64_t)c->pool_of[x] * c->slot_bytes);
        }
        if (!c->io_keys.empty()) {
          s = store_submit(c->kv_store, c->io_keys.data(), (int64_t)c->io_keys.size(), c->io_dst.data(),
                           &a.ticket);
          if (s != CKV_OK) return s;
          stv.bytes_storage += (int64_t)c->io_keys.size() * c->slot_bytes;
        }
      }
    }
    if ((s = demand_and_attention()) != CKV_OK) return s;
  }

  if (nf > 0) {  // chunks entering the GPU tier, after the attention that read their slots
    CKV_HIP(hipMemcpyAsync(c->fill_dev[cur], c->fill_host[cur], (size_t)(2 * k) * sizeof(int32_t),
                           hipMemcpyHostToDevice, st));
    s = launch_copy_slots(c->arena, c->fill_dev[cur], c->arena, c->fill_dev[cur] + k, nf,
                          c->slot_bytes, st);
    if (s != CKV_OK) return s;
    stv.bytes_cache_fill = nf * c->slot_bytes;
  }
  // after the cache fills too: they read this layer's buffer
  CKV_HIP(hipEventRecord(c->ev_attn[cur], st));
  c->attn_recorded[cur] = true;

  if (has_next && !stored) {  // the next layer's copy, over the host link on the side stream
    if (c->attn_recorded[nxt]) CKV_HIP(hipStreamWaitEvent(c->prefetch, c->ev_attn[nxt], 0));
    // after this layer's demand copies: those are on the critical path and get
    // the host link to themselves
    CKV_HIP(hipStreamWaitEvent(c->prefetch, c->ev_dem, 0));
    if (np > 0) {
      std::memcpy(c->pref_host[nxt], c->pred.data(), (size_t)np * sizeof(int32_t));
      CKV_HIP(hipMemcpyAsync(c->pref_dev[nxt], c->pref_host[nxt], (size_t)np * sizeof(int32_t),
                             hipMemcpyHostToDevice, c->prefetch));
      s = launch_copy_spans(store_next, c->pref_dev[nxt], np, 0, c->slots[nxt], c->slot_bytes,
                            c->prefetch);
      if (s != CKV_OK) return s;
    }
    CKV_HIP(hipEventRecord(c->ev_pref[nxt], c->prefetch));
    c->pref_pending[nxt] = true;
    c->pref_recorded[nxt] = true;
  }
  c->next_layer = layer + 1;
  if (stats) *stats = stv;
  return CKV_OK;
}

}  // extern "C"
