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
// Host-resident prefix (Sec. 4.3.2): the K/V store of every layer lives in
// pinned host memory, chunk-major (chunk j of a layer is one span: K rows then
// V rows).  HBM holds a ring of transient slot buffers, layer l using buffer
// l % nbuf.  Chunks predicted for a layer are copied into its buffer ahead of
// time on a prefetch stream (the prediction P_{l+1} = S_l, or a set the caller
// gives); when the layer has selected S_l only the difference S_l \ P_l is
// fetched on a demand stream into the free slots behind the predicted ones,
// and the attention reads every kept chunk through a chunk -> slot table: it
// attends over the chunks already in HBM while the misses are copied, and
// over each share of the misses once that share's copy has landed (bf16).
// With Periods and the per-layer stores registered (ckv_ctx_set_host_layers),
// a Period's first layer queues the copies of every later layer of its Period
// as soon as its set is known (intra-period prefetch; the ring then holds
// p + 1 buffers), and its attention waits until the first `subperiod` layers
// of the Period are in HBM (SubPeriod gating).  Copies move whole chunk spans,
// by a kernel that reads the pinned store over the host link.  The selection
// is the step's only device -> host dependency.
//
// Pinned staging lists (slot tables, chunk lists) are rewritten only after
// the copy that last read them has run: every staging copy records a guard
// event that the host waits on before the next rewrite.

#include <cstring>
#include <new>
#include <vector>

#include "tiers_internal.h"

using namespace ckv;

namespace {

constexpr int kMaxBuf = 17;  // Periods of up to 16 layers, plus the next Period's first layer

// One transient slot buffer: slots_per_buf chunk slots of the arena and the
// staging of the layer that uses it.
struct SlotBuf {
  void* slots = nullptr;
  // device lists and their pinned staging: chunk -> arena slot table [k],
  // demand chunks [k], prefetch chunks [k], cache fills [2k] (source slots,
  // then target slots)
  int32_t *tab_dev = nullptr, *tab_host = nullptr;
  int32_t *dem_dev = nullptr, *dem_host = nullptr;
  int32_t *pref_dev = nullptr, *pref_host = nullptr;
  int32_t *fill_dev = nullptr, *fill_host = nullptr;
  hipEvent_t ev_pref = nullptr;  // the copies into this buffer's predicted slots have landed
  hipEvent_t ev_attn = nullptr;  // the last layer reading this buffer (attention, fills) is done
  // staging guards: recorded after the staging copies of tab/dem (demand
  // stream), pref (prefetch stream) and fill (compute stream)
  hipEvent_t ev_gd = nullptr, ev_gp = nullptr, ev_gf = nullptr;
  bool pref_pending = false, attn_rec = false, gd = false, gp = false, gf = false;
  int32_t pred_layer = -1;      // layer whose predicted chunks sit in slots 0..|pred|-1
  std::vector<int32_t> pred;    // those chunks, ascending
};

}  // namespace

struct ckv_ctx {
  ckv_dims dims;
  int32_t n_layers;
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
  // one arena of chunk slots: nbuf transient buffers of slots_per_buf slots,
  // then cache_slots slots holding the chunks of an attached cache's GPU tier;
  // slot tables index the whole arena
  int nbuf = 2;
  void* arena = nullptr;
  SlotBuf buf[kMaxBuf];
  int32_t* stage_host = nullptr;  // pinned staging of every buffer (5k ints each)
  int32_t* stage_dev = nullptr;
  int32_t* sel_host = nullptr;    // pinned [k]
  hipStream_t demand = nullptr, prefetch = nullptr;
  hipEvent_t ev_sel = nullptr, ev_dem = nullptr;
  hipEvent_t ev_tab = nullptr;  // the attention lists of the layer are on the device
  // host-resident bf16 layers attend in parts: the chunks already in HBM with
  // the suffix, then each of up to kLateParts shares of the chunks copied on
  // demand once its copy has landed (ev_late[i]; the storage tier's one copy
  // out of its pool lands every share).  attn_splits: the most splits the
  // parts take
  static constexpr int kLateParts = 4;
  hipEvent_t ev_late[kLateParts] = {};
  int64_t attn_splits = 0;
  std::vector<int32_t> slot_sorted;  // arena slot of each kept chunk, ascending chunk order
  std::vector<const void*> host_layers;  // device views of the registered per-layer stores
  int32_t prev_layer = -1;  // last layer run since creation or reset (-1: none)
  bool broken = false;      // a layer failed after enqueueing work: reset before the next
  int32_t inject_layer = -1;  // test hook: the demand copy of this layer fails
  // Periods: layers period_first .. period_first+period-1 attend over the set
  // selected at period_first (device copy at off_pset, host copy pset_host)
  int32_t period = 1;
  int32_t period_first = -1;  // -1: no set held
  int32_t subperiod = 1;
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
  double* scores_host = nullptr;    // pinned [m]
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
  std::vector<int64_t> io_keys, dropped;
  std::vector<char*> io_dst;
  std::vector<int32_t> xsrc, xdst;
  // stage timing: a ring of event sets, harvested when a set is reused or on query
  static constexpr int kRing = 64;
  hipEvent_t tev[kRing][CKV_N_STAGES + 1] = {};
  int64_t t_issued = 0, t_done = 0;
  double t_ms[CKV_N_STAGES] = {};
  // scoring-kernel timing (bf16): per scored layer, every workgroup's start
  // and end from the realtime counter (span_words per layer), in a device ring
  static constexpr int kSpanRing = 1024;
  unsigned long long* tspan = nullptr;  // [kSpanRing][span_words]
  int64_t span_words = 0;
  bool span_mode = false;
};

namespace {

// Waits for the copy that last read a pinned staging list before it is rewritten.
ckv_status guard(hipEvent_t e, bool& recorded) {
  if (recorded) {
    CKV_HIP(hipEventSynchronize(e));
    recorded = false;
  }
  return CKV_OK;
}

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
// with the lists staged through this buffer's pinned and device arrays; the
// staging guard of that stream is recorded after the list copy.
ckv_status pool_copy(ckv_ctx* c, int b, int which, const int32_t* src, const int32_t* dst,
                     int64_t count, hipStream_t st) {
  if (count == 0) return CKV_OK;
  SlotBuf& B = c->buf[b];
  ckv_status s = which == 0 ? guard(B.ev_gp, B.gp) : guard(B.ev_gd, B.gd);
  if (s != CKV_OK) return s;
  const int64_t spb = c->slots_per_buf;
  int32_t* h = c->xfer_host[b][which];
  std::memcpy(h, src, (size_t)count * sizeof(int32_t));
  std::memcpy(h + spb, dst, (size_t)count * sizeof(int32_t));
  CKV_HIP(hipMemcpyAsync(c->xfer_dev[b][which], h, (size_t)(2 * spb) * sizeof(int32_t),
                         hipMemcpyHostToDevice, st));
  if (which == 0) {
    CKV_HIP(hipEventRecord(B.ev_gp, st));
    B.gp = true;
  } else {
    CKV_HIP(hipEventRecord(B.ev_gd, st));
    B.gd = true;
  }
  return launch_copy_slots(c->pool_dev, c->xfer_dev[b][which], c->arena,
                           c->xfer_dev[b][which] + spb, count, c->slot_bytes, st);
}

void free_buffers(ckv_ctx* c) {
  for (SlotBuf& B : c->buf) {
    for (hipEvent_t e : {B.ev_pref, B.ev_attn, B.ev_gd, B.ev_gp, B.ev_gf})
      if (e) (void)hipEventDestroy(e);
    B = SlotBuf();
  }
  (void)hipHostFree(c->stage_host);
  (void)hipFree(c->stage_dev);
  c->stage_host = nullptr;
  c->stage_dev = nullptr;
}

ckv_status free_ctx(ckv_ctx* c) {
  if (!c) return CKV_OK;
  drain_store_reads(c);
  if (c->cache) cache_log_gpu_evictions(c->cache, false);  // the cache outlives the context
  if (c->demand) (void)hipStreamSynchronize(c->demand);
  if (c->prefetch) (void)hipStreamSynchronize(c->prefetch);
  (void)hipFree(c->ws);
  free_buffers(c);
  (void)hipFree(c->arena);
  free_pool(c);
  (void)hipHostFree(c->sel_host);
  (void)hipHostFree(c->scores_host);
  for (auto& set : c->tev)
    for (auto& e : set)
      if (e) (void)hipEventDestroy(e);
  (void)hipFree(c->tspan);
  if (c->ev_sel) (void)hipEventDestroy(c->ev_sel);
  if (c->ev_dem) (void)hipEventDestroy(c->ev_dem);
  if (c->ev_tab) (void)hipEventDestroy(c->ev_tab);
  for (hipEvent_t e : c->ev_late)
    if (e) (void)hipEventDestroy(e);
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

// Staging of every slot buffer: one pinned and one device block of kMaxBuf *
// 5k ints, carved per buffer, and the buffers' events.
ckv_status alloc_buffers(ckv_ctx* c) {
  const size_t per = (size_t)(5 * c->k);
  const size_t bytes = per * kMaxBuf * sizeof(int32_t);
  hipError_t e = hipHostMalloc((void**)&c->stage_host, bytes, hipHostMallocDefault);
  if (e == hipSuccess) e = hipMalloc((void**)&c->stage_dev, bytes);
  for (int b = 0; b < kMaxBuf && e == hipSuccess; ++b) {
    SlotBuf& B = c->buf[b];
    int32_t* h = c->stage_host + b * per;
    int32_t* d = c->stage_dev + b * per;
    B.tab_host = h;
    B.tab_dev = d;
    B.dem_host = h + c->k;
    B.dem_dev = d + c->k;
    B.pref_host = h + 2 * c->k;
    B.pref_dev = d + 2 * c->k;
    B.fill_host = h + 3 * c->k;
    B.fill_dev = d + 3 * c->k;
    for (hipEvent_t* ev : {&B.ev_pref, &B.ev_attn, &B.ev_gd, &B.ev_gp, &B.ev_gf})
      if (e == hipSuccess) e = hipEventCreateWithFlags(ev, hipEventDisableTiming);
  }
  if (e != hipSuccess)
    CKV_FAIL(e == hipErrorOutOfMemory ? CKV_ENOMEM : CKV_EHIP, "slot buffer staging: %s",
             hipGetErrorString(e));
  return CKV_OK;
}

// (Re)allocates the slot arena for nbuf transient buffers and G cache slots;
// with keep_cache, the bytes of the current G cache slots move to the new
// arena (the chunks of an attached cache's GPU tier stay in HBM).  The device
// must be idle (nothing in flight may read the old arena).
ckv_status alloc_arena(ckv_ctx* c, int nbuf, int64_t G, bool keep_cache = false) {
  const size_t bytes = (size_t)((nbuf * c->slots_per_buf + G) * c->slot_bytes);
  void* arena = nullptr;
  hipError_t e = hipMalloc(&arena, bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    CKV_FAIL(e == hipErrorOutOfMemory ? CKV_ENOMEM : CKV_EHIP,
             "hipMalloc of %zu bytes of chunk slots failed: %s", bytes, hipGetErrorString(e));
  }
  if (keep_cache && c->arena && G > 0 && G == c->cache_slots) {
    e = hipMemcpy(static_cast<char*>(arena) + nbuf * c->slots_per_buf * c->slot_bytes,
                  static_cast<char*>(c->arena) + c->nbuf * c->slots_per_buf * c->slot_bytes,
                  (size_t)(G * c->slot_bytes), hipMemcpyDeviceToDevice);
    if (e != hipSuccess) {
      (void)hipFree(arena);
      CKV_FAIL(CKV_EHIP, "moving the cache slots to the new arena failed: %s", hipGetErrorString(e));
    }
  }
  CKV_HIP(hipFree(c->arena));
  c->arena = arena;
  c->nbuf = nbuf;
  for (int b = 0; b < kMaxBuf; ++b) {
    SlotBuf& B = c->buf[b];
    B.slots = b < nbuf ? static_cast<char*>(arena) + b * c->slots_per_buf * c->slot_bytes : nullptr;
    B.pred_layer = -1;
    B.pred.clear();
    B.pref_pending = false;
    B.attn_rec = false;
  }
  return CKV_OK;
}

// Ring size the current settings call for: a Period's layers plus the next
// Period's first layer when intra-period prefetch is possible (pinned stores
// registered, no storage tier, 1 < p < kMaxBuf), else two buffers.
int wanted_buffers(const ckv_ctx* c) {
  if (!(c->flags & CKV_CTX_HOST_PREFIX) || c->kv_store || c->host_layers.empty()) return 2;
  if (c->period <= 1 || c->period + 1 > kMaxBuf) return 2;
  return c->period + 1;
}

bool period_wide(const ckv_ctx* c) { return c->nbuf > 2; }

ckv_status resize_ring(ckv_ctx* c) {
  const int nb = wanted_buffers(c);
  if (nb == c->nbuf) return CKV_OK;
  CKV_HIP(hipDeviceSynchronize());
  return alloc_arena(c, nb, c->cache_slots, true);
}

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

// Ticks of the realtime counter the scoring kernel's spans are measured in.
constexpr double kRealtimeTickMs = 1e-5;  // 100 MHz

// Adds the span (earliest workgroup start to latest end) of every scored
// layer not yet accounted; waits for the device.
ckv_status harvest_spans(ckv_ctx* c) {
  if (c->t_done == c->t_issued) return CKV_OK;
  CKV_HIP(hipDeviceSynchronize());
  const int64_t wpl = c->span_words;
  std::vector<unsigned long long> h((size_t)(wpl * ckv_ctx::kSpanRing));
  CKV_HIP(hipMemcpy(h.data(), c->tspan, h.size() * sizeof(unsigned long long),
                    hipMemcpyDeviceToHost));
  for (int64_t i = c->t_done; i < c->t_issued; ++i) {
    const unsigned long long* t = h.data() + (i % ckv_ctx::kSpanRing) * wpl;
    unsigned long long t0 = ~0ull, t1 = 0;
    for (int64_t w = 0; w < wpl; w += 2) {
      t0 = std::min(t0, t[w]);
      t1 = std::max(t1, t[w + 1]);
    }
    if (t1 > t0) c->t_ms[CKV_STAGE_SCORE] += (double)(t1 - t0) * kRealtimeTickMs;
  }
  c->t_done = c->t_issued;
  return CKV_OK;
}

ckv_status harvest_all(ckv_ctx* c) {
  if (c->span_mode) return harvest_spans(c);
  while (c->t_done < c->t_issued) {
    ckv_status s = harvest_one(c);
    if (s != CKV_OK) return s;
  }
  return CKV_OK;
}

int64_t chunk_len(const ckv_dims* d, int64_t j) {
  return std::min<int64_t>(d->chunk_size, d->n_prefix - j * d->chunk_size);
}

int64_t chunk_bytes(const ckv_ctx* c, int64_t j) {
  const ckv_dims* d = &c->dims;
  return 2 * chunk_len(d, j) * d->n_kv_heads * d->head_dim * elem_bytes(d->dtype);
}

// Queues, on the prefetch stream, the copy of `chunks` (ascending) of layer
// t's pinned store into slots 0.. of buffer b, after the layer that last read
// the buffer and after this layer's demand copies; the buffer then predicts
// layer t.  Returns the bytes queued.
ckv_status queue_prefetch(ckv_ctx* c, int b, int32_t t, const void* store,
                          const std::vector<int32_t>& chunks, bool after_demand, int64_t* bytes) {
  SlotBuf& B = c->buf[b];
  if (B.attn_rec) CKV_HIP(hipStreamWaitEvent(c->prefetch, B.ev_attn, 0));
  if (after_demand) CKV_HIP(hipStreamWaitEvent(c->prefetch, c->ev_dem, 0));
  const int64_t n = (int64_t)chunks.size();
  if (n > 0) {
    ckv_status s = guard(B.ev_gp, B.gp);
    if (s != CKV_OK) return s;
    std::memcpy(B.pref_host, chunks.data(), (size_t)n * sizeof(int32_t));
    CKV_HIP(hipMemcpyAsync(B.pref_dev, B.pref_host, (size_t)n * sizeof(int32_t),
                           hipMemcpyHostToDevice, c->prefetch));
    CKV_HIP(hipEventRecord(B.ev_gp, c->prefetch));
    B.gp = true;
    s = launch_copy_spans(store, B.pref_dev, n, 0, B.slots, c->slot_bytes, c->prefetch);
    if (s != CKV_OK) return s;
  }
  CKV_HIP(hipEventRecord(B.ev_pref, c->prefetch));
  B.pref_pending = true;
  B.pred = chunks;
  B.pred_layer = t;
  for (int32_t j : chunks) *bytes += chunk_bytes(c, j);
  return CKV_OK;
}

// The chunks of `set` that layer t does not find in the attached cache's HBM slots.
void uncached(const ckv_ctx* c, int32_t t, const int32_t* set, int64_t n, std::vector<int32_t>& out) {
  out.clear();
  const bool t_cached = c->cache && t < c->cache_layers;
  const int64_t key0 = (int64_t)t * c->m;
  for (int64_t u = 0; u < n; ++u)
    if (!(t_cached && c->slot_of[key0 + set[u]] >= 0)) out.push_back(set[u]);
}

struct LayerArgs {
  int32_t layer;
  const ckv_layer_io* io;
  const void* store;       // this layer's pinned store as the device reads it
  const void* store_next;  // the next layer's, or nullptr
  bool explicit_pred;
};

ckv_status run_layer(ckv_ctx* c, const LayerArgs& la, ckv_layer_stats* stats);

}  // namespace

extern "C" {

ckv_status ckv_ctx_create(const ckv_dims* dims, int32_t n_layers, double keep_ratio, int32_t flags,
                          ckv_ctx** out) {
  clear_error();
  if (!out) CKV_FAIL(CKV_EINVAL, "out is NULL");
  *out = nullptr;
  {
    ckv_status s = check_dims(dims);
    if (s != CKV_OK) return s;
  }
  if (n_layers < 1) CKV_FAIL(CKV_EINVAL, "n_layers must be >= 1 (got %d)", n_layers);
  if (!(keep_ratio > 0.0 && keep_ratio <= 1.0)) CKV_FAIL(CKV_EINVAL, "keep_ratio must be in (0, 1]");
  if (flags & ~(CKV_CTX_HOST_PREFIX | CKV_CTX_MATERIALIZE | CKV_CTX_STAGE_TIMING |
                CKV_CTX_SCORE_TIMING))
    CKV_FAIL(CKV_EINVAL, "unknown flags");
  ckv_ctx* c = new (std::nothrow) ckv_ctx();
  if (!c) CKV_FAIL(CKV_ENOMEM, "host allocation failed");
  c->dims = *dims;
  c->n_layers = n_layers;
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
  if ((flags & CKV_CTX_HOST_PREFIX) && dims->dtype == CKV_DTYPE_BF16) {
    c->attn_splits = attn_parted_splits(dims, c->k, ckv_ctx::kLateParts);
    c->ws_attn = std::max(c->ws_attn, attn_parted_bytes(dims, c->attn_splits));
  }
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
    ckv_status s = alloc_buffers(c);
    if (s == CKV_OK) s = alloc_arena(c, 2, 0);
    if (s != CKV_OK) {
      free_ctx(c);
      return s;
    }
    CKV_HIP_ALLOC(hipHostMalloc((void**)&c->sel_host, (size_t)c->k * sizeof(int32_t),
                                hipHostMallocDefault));
    CKV_HIP_ALLOC(hipHostMalloc((void**)&c->scores_host, (size_t)c->m * sizeof(double),
                                hipHostMallocDefault));
    CKV_HIP_ALLOC(hipStreamCreateWithFlags(&c->demand, hipStreamNonBlocking));
    CKV_HIP_ALLOC(hipStreamCreateWithFlags(&c->prefetch, hipStreamNonBlocking));
    CKV_HIP_ALLOC(hipEventCreateWithFlags(&c->ev_sel, hipEventDisableTiming));
    CKV_HIP_ALLOC(hipEventCreateWithFlags(&c->ev_dem, hipEventDisableTiming));
    CKV_HIP_ALLOC(hipEventCreateWithFlags(&c->ev_tab, hipEventDisableTiming));
    for (hipEvent_t& e : c->ev_late) CKV_HIP_ALLOC(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  }
  c->span_mode = (flags & CKV_CTX_SCORE_TIMING) && !(flags & CKV_CTX_STAGE_TIMING) &&
                 dims->dtype == CKV_DTYPE_BF16;
  if (c->span_mode) {
    c->span_words = score_span_words(dims);
    CKV_HIP_ALLOC(hipMalloc((void**)&c->tspan, (size_t)(c->span_words * ckv_ctx::kSpanRing) *
                                                   sizeof(unsigned long long)));
  } else if (flags & (CKV_CTX_STAGE_TIMING | CKV_CTX_SCORE_TIMING)) {
    for (auto& set : c->tev)
      for (auto& e : set) CKV_HIP_ALLOC(hipEventCreate(&e));
  }
  *out = c;
  return CKV_OK;
}

ckv_status ckv_ctx_stage_times(ckv_ctx* ctx, double* ms, int64_t* n_layers) {
  clear_error();
  if (!ctx || !ms || !n_layers) CKV_FAIL(CKV_EINVAL, "NULL argument");
  if (!(ctx->flags & (CKV_CTX_STAGE_TIMING | CKV_CTX_SCORE_TIMING)))
    CKV_FAIL(CKV_ESTATE, "context created without CKV_CTX_STAGE_TIMING or CKV_CTX_SCORE_TIMING");
  {
    ckv_status s = harvest_all(ctx);
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
  const int old = ctx->period;
  ctx->period = period;
  if (wanted_buffers(ctx) != ctx->nbuf) {
    if (ctx->prev_layer >= 0) {
      ctx->period = old;
      CKV_FAIL(CKV_ESTATE, "with registered host stores, set the Period at the start of a request");
    }
    ckv_status s = resize_ring(ctx);
    if (s != CKV_OK) {
      ctx->period = old;
      return s;
    }
  }
  ctx->period_first = -1;
  return CKV_OK;
}

ckv_status ckv_ctx_set_host_layers(ckv_ctx* ctx, const void* const* kv_host, int32_t n) {
  clear_error();
  if (!ctx) CKV_FAIL(CKV_EINVAL, "ctx is NULL");
  if (!(ctx->flags & CKV_CTX_HOST_PREFIX))
    CKV_FAIL(CKV_EINVAL, "host stores need a context with a host-resident prefix");
  if (ctx->prev_layer >= 0)
    CKV_FAIL(CKV_ESTATE, "register host stores at the start of a request (before its first layer)");
  std::vector<const void*> views;
  if (kv_host) {
    if (n != ctx->n_layers)
      CKV_FAIL(CKV_EINVAL, "%d host stores for a context of %d layers", n, ctx->n_layers);
    views.resize((size_t)n);
    for (int32_t l = 0; l < n; ++l) {
      views[l] = kv_host[l] ? device_view(kv_host[l]) : nullptr;
      if (!views[l])
        CKV_FAIL(CKV_EINVAL, "host store of layer %d is not pinned host memory (hipHostMalloc)", l);
    }
  }
  std::swap(ctx->host_layers, views);
  ckv_status s = resize_ring(ctx);
  if (s != CKV_OK) std::swap(ctx->host_layers, views);
  return s;
}

ckv_status ckv_ctx_inject_copy_error(ckv_ctx* ctx, int32_t layer) {
  clear_error();
  if (!ctx) CKV_FAIL(CKV_EINVAL, "ctx is NULL");
  if (!(ctx->flags & CKV_CTX_HOST_PREFIX))
    CKV_FAIL(CKV_EINVAL, "copy errors are injected on a host-resident prefix only");
  if (layer < -1 || layer >= ctx->n_layers)
    CKV_FAIL(CKV_EINVAL, "layer must be -1 or in [0, %d)", ctx->n_layers);
  ctx->inject_layer = layer;
  return CKV_OK;
}

ckv_status ckv_ctx_attach_cache(ckv_ctx* ctx, ckv_cache* cache) {
  clear_error();
  if (!ctx) CKV_FAIL(CKV_EINVAL, "ctx is NULL");
  if (!(ctx->flags & CKV_CTX_HOST_PREFIX))
    CKV_FAIL(CKV_EINVAL, "a cache needs a context with a host-resident prefix");
  if (ctx->prev_layer >= 0)
    CKV_FAIL(CKV_ESTATE, "attach a cache at the start of a request (before its first layer or after a reset)");
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
    if (kMaxBuf * ctx->slots_per_buf + G > INT32_MAX)
      CKV_FAIL(CKV_EUNSUPPORTED, "too many cache slots (%lld)", (long long)G);
  }
  // the arena is replaced with nothing in flight that could still read it
  CKV_HIP(hipDeviceSynchronize());
  ckv_status s = alloc_arena(ctx, ctx->nbuf, G);
  if (s != CKV_OK) return s;
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
  if (ctx->prev_layer >= 0)
    CKV_FAIL(CKV_ESTATE, "attach a store at the start of a request (before its first layer or after a reset)");
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
  if (!store) return resize_ring(ctx);
  // room for the cache's tiers, plus the transient chunks of two layers in
  // flight and of the layer whose slots wait for release.  With few keys the
  // count is capped at one slot per key plus the quarantine: a layer releases
  // at most 3k slots (its set, its unused prediction and the chunks the
  // cascade dropped), and a key released that way can take a second slot for
  // the next layer's reads while its old one still waits
  const int64_t keys = store_keys(store), k = ctx->k;
  const int64_t kept = ctx->cache ? std::min(keys, cache_gpu_slots(ctx->cache) + cache_cpu_slots(ctx->cache)) : 0;
  const int64_t n = std::min(keys + 3 * k, kept + (6 + ctx->subperiod) * k) + 16;
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
  return resize_ring(ctx);  // the storage tier runs on two buffers
}

ckv_status ckv_ctx_reset(ckv_ctx* ctx) {
  clear_error();
  if (!ctx) CKV_FAIL(CKV_EINVAL, "ctx is NULL");
  if (ctx->prefetch) CKV_HIP(hipStreamSynchronize(ctx->prefetch));
  if (ctx->demand) CKV_HIP(hipStreamSynchronize(ctx->demand));
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
  for (SlotBuf& B : ctx->buf) {
    B.pred_layer = -1;
    B.pred.clear();
    B.pref_pending = false;
  }
  ctx->prev_layer = -1;
  ctx->period_first = -1;
  ctx->broken = false;
  ctx->inject_layer = -1;
  {
    ckv_status s = harvest_all(ctx);
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
  if (c->broken)
    CKV_FAIL(CKV_ESTATE, "an earlier layer failed after enqueueing work: reset the context first");
  const bool host = c->flags & CKV_CTX_HOST_PREFIX;
  if (layer < 0 || layer >= c->n_layers)
    CKV_FAIL(CKV_EINVAL, "layer must be in [0, %d) (got %d)", c->n_layers, layer);
  if (!io->q || !io->k_suffix || !io->v_suffix || !io->k_probe || !io->out)
    CKV_FAIL(CKV_EINVAL, "NULL tensor in io");
  if (!aligned16(io->q) || !aligned16(io->k_suffix) || !aligned16(io->v_suffix) ||
      !aligned16(io->k_probe) || !aligned16(io->out))
    CKV_FAIL(CKV_EINVAL, "tensors must be 16-byte aligned");
  LayerArgs la{layer, io, nullptr, nullptr, io->pred_idx != nullptr};
  if (la.explicit_pred) {
    if (io->n_pred < 0 || io->n_pred > c->k)
      CKV_FAIL(CKV_EINVAL, "n_pred must be in [0, k = %lld] (got %lld)", (long long)c->k,
               (long long)io->n_pred);
    for (int64_t u = 0; u < io->n_pred; ++u) {
      const int32_t j = io->pred_idx[u];
      if (j < 0 || j >= c->m || (u > 0 && j <= io->pred_idx[u - 1]))
        CKV_FAIL(CKV_EINVAL, "pred_idx must be strictly ascending chunk indices in [0, %lld)",
                 (long long)c->m);
    }
  }
  const bool stored = host && c->kv_store;  // chunks come from the storage tier
  if (host) {
    if (c->prev_layer >= 0 && layer != c->prev_layer + 1)
      CKV_FAIL(CKV_ESTATE, "host-resident layers must run in order (expected %d, got %d)",
               c->prev_layer + 1, layer);
  }
  if (stored) {
    if (layer >= c->store_layers)
      CKV_FAIL(CKV_EINVAL, "layer %d is not in the attached store (%lld layers)", layer,
               (long long)c->store_layers);
    if (la.explicit_pred)
      CKV_FAIL(CKV_EUNSUPPORTED, "a caller prediction with an attached store is not supported");
  } else if (host) {
    // the copy kernels read the stores through the device's mapping of them
    if (io->kv_host) {
      la.store = device_view(io->kv_host);
      if (!la.store) CKV_FAIL(CKV_EINVAL, "kv_host must be pinned host memory (hipHostMalloc)");
    } else if (!c->host_layers.empty()) {
      la.store = c->host_layers[layer];
    } else {
      CKV_FAIL(CKV_EINVAL, "host-resident prefix needs kv_host (or registered host stores)");
    }
    if (!c->host_layers.empty()) {
      la.store_next = layer + 1 < c->n_layers ? c->host_layers[layer + 1] : nullptr;
    } else if (io->kv_host_next && layer + 1 < c->n_layers) {
      la.store_next = device_view(io->kv_host_next);
      if (!la.store_next) CKV_FAIL(CKV_EINVAL, "kv_host_next must be pinned host memory (hipHostMalloc)");
    }
  } else {
    if (!io->k_prefix || !io->v_prefix) CKV_FAIL(CKV_EINVAL, "HBM-resident prefix needs k/v_prefix");
    if (!aligned16(io->k_prefix) || !aligned16(io->v_prefix))
      CKV_FAIL(CKV_EINVAL, "tensors must be 16-byte aligned");
  }
  if (host && c->cache && layer >= c->cache_layers)
    CKV_FAIL(CKV_EINVAL, "layer %d has no keys in the attached cache (%lld layers)", layer,
             (long long)c->cache_layers);
  // a layer past the first of its Period reuses the set selected there
  const int32_t first = layer - layer % c->period;
  if (first != layer && c->period_first != first)
    CKV_FAIL(CKV_ESTATE, "layer %d reuses the set of layer %d, the first of its Period, which has not run",
             layer, first);
  const ckv_status s = run_layer(c, la, stats);
  if (s != CKV_OK) c->broken = true;
  return s;
}

}  // extern "C"

namespace {

ckv_status run_layer(ckv_ctx* c, const LayerArgs& la, ckv_layer_stats* stats) {
  const ckv_layer_io* io = la.io;
  const int32_t layer = la.layer;
  const ckv_dims* d = &c->dims;
  const bool host = c->flags & CKV_CTX_HOST_PREFIX;
  const bool stored = host && c->kv_store;
  const int32_t first = layer - layer % c->period;
  const bool reuse = first != layer;
  hipStream_t st = (hipStream_t)io->stream;
  char* ws = static_cast<char*>(c->ws);
  double* scores = io->chunk_scores ? io->chunk_scores : reinterpret_cast<double*>(ws + c->off_scores);
  int32_t* pset = reinterpret_cast<int32_t*>(ws + c->off_pset);
  // the set this layer attends over: selected now, or the Period's
  int32_t* sel = reuse ? pset : io->sel_idx ? io->sel_idx : reinterpret_cast<int32_t*>(ws + c->off_sel);
  const int64_t k = c->k;
  const int eb = elem_bytes(d->dtype);
  const int64_t span_elems = (int64_t)d->chunk_size * d->n_kv_heads * d->head_dim;
  ckv_layer_stats stv{};
  stv.k = k;
  ckv_status s = CKV_OK;

  // a caller prediction for this pinned-host layer: its copy goes out first,
  // beside this layer's scoring
  const int cur = host ? layer % c->nbuf : 0;
  if (host && !stored && la.explicit_pred) {
    std::vector<int32_t> P;
    uncached(c, layer, io->pred_idx, io->n_pred, P);
    s = queue_prefetch(c, cur, layer, la.store, P, false, &stv.bytes_prefetch);
    if (s != CKV_OK) return s;
  }

  hipEvent_t* tev = nullptr;
  unsigned long long* span = nullptr;
  // a reused layer has no scoring kernel to time alone
  if (c->span_mode) {
    if (!reuse) {
      if (c->t_issued - c->t_done >= ckv_ctx::kSpanRing) {  // ring full: account it first
        s = harvest_spans(c);
        if (s != CKV_OK) return s;
      }
      span = c->tspan + c->span_words * (c->t_issued % ckv_ctx::kSpanRing);
    }
  } else if ((c->flags & CKV_CTX_STAGE_TIMING) || ((c->flags & CKV_CTX_SCORE_TIMING) && !reuse)) {
    if (c->t_issued - c->t_done >= ckv_ctx::kRing) {  // reuse the oldest set: account it first
      s = harvest_one(c);
      if (s != CKV_OK) return s;
    }
    tev = c->tev[c->t_issued % ckv_ctx::kRing];
    CKV_HIP(hipEventRecord(tev[0], st));  // the set starts here
  }
  auto mark = [&](int i) -> ckv_status {
    if (tev && all_stages(c)) CKV_HIP(hipEventRecord(tev[i], st));
    return CKV_OK;
  };

  if (!reuse) {
    s = launch_score(d, io->q, io->k_probe, scores, ws, c->ws_score, st, tev ? tev[1] : nullptr,
                     span);
    if (s != CKV_OK) return s;
    if (span) ++c->t_issued;
    if ((s = mark(2)) != CKV_OK) return s;
    // with Periods the selection also keeps the set for the rest of the Period
    s = launch_select(scores, c->m, k, sel, nullptr, 0, st, c->period > 1 ? pset : nullptr);
    if (s != CKV_OK) return s;
    if ((s = mark(3)) != CKV_OK) return s;
    if (c->period > 1) c->period_first = layer;
  } else {
    if ((s = mark(1)) != CKV_OK) return s;
    if ((s = mark(2)) != CKV_OK) return s;
    if (io->sel_idx)  // the caller sees the set the layer used
      CKV_HIP(hipMemcpyAsync(io->sel_idx, pset, (size_t)k * sizeof(int32_t),
                             hipMemcpyDeviceToDevice, st));
    if ((s = mark(3)) != CKV_OK) return s;
  }

  if (!host) {
    ChunkSource src{io->k_prefix, io->v_prefix, span_elems, nullptr, 1, c->m};
    if (c->flags & CKV_CTX_MATERIALIZE) {
      void* ksel = ws + c->off_ksel;
      void* vsel = ws + c->off_vsel;
      s = launch_gather(d, io->k_prefix, io->v_prefix, sel, k, ksel, vsel, st);
      if (s != CKV_OK) return s;
      src = ChunkSource{ksel, vsel, span_elems, nullptr, 0, k};
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
    c->prev_layer = layer;
    if (stats) *stats = stv;
    return CKV_OK;
  }

  // ---- host-resident prefix ------------------------------------------------
  SlotBuf& B = c->buf[cur];
  const bool cached = c->cache != nullptr;
  const int64_t key0 = (int64_t)layer * c->m;
  const int64_t spb = c->slots_per_buf;
  const int64_t buf0 = cur * spb, cache0 = c->nbuf * spb;
  ckv_ctx::Ahead& mine = c->ahead[layer % ckv_ctx::kAhead];
  std::vector<int32_t> P;  // this layer's predicted chunks, in slots 0..|P|-1 of its buffer
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
    // a predicted chunk whose pool slot was released since it was listed (the
    // cache sent it out of memory at an intervening layer) is fetched on
    // demand like any miss
    c->xsrc.clear();
    c->xdst.clear();
    for (size_t i = 0; i < mine.chunks.size(); ++i) {
      const int32_t sl = c->pool_of[mine.keys[i]];
      if (sl < 0) continue;
      c->xsrc.push_back(sl);
      c->xdst.push_back((int32_t)(buf0 + P.size()));
      P.push_back(mine.chunks[i]);
    }
    if (!P.empty()) {
      // the predicted chunks move to this layer's HBM slots 0..|P|-1 on the
      // prefetch stream, beside this layer's scoring
      if (B.attn_rec) CKV_HIP(hipStreamWaitEvent(c->prefetch, B.ev_attn, 0));
      CKV_HIP(hipStreamWaitEvent(c->prefetch, c->ev_dem, 0));
      s = pool_copy(c, cur, 0, c->xsrc.data(), c->xdst.data(), (int64_t)P.size(), c->prefetch);
      if (s != CKV_OK) return s;
      CKV_HIP(hipEventRecord(B.ev_pref, c->prefetch));
      B.pref_pending = true;
    }
  } else if (B.pred_layer == layer) {
    P = B.pred;
  }
  if (reuse) {  // the Period's set is already on the host: no synchronisation
    if (stored) {
      // pool slots released by the previous layer are reused below: its copies
      // out of them must have finished
      const SlotBuf& Bn = c->buf[(layer + c->nbuf - 1) % c->nbuf];
      if (Bn.attn_rec) CKV_HIP(hipEventSynchronize(Bn.ev_attn));
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

  // slot of each kept chunk, in arena slots: chunks held in the cache's HBM
  // slots are read there; predicted chunks sit in this layer's buffer at slots
  // 0..|P|-1 (in P order), misses follow
  if ((s = guard(B.ev_gd, B.gd)) != CKV_OK) return s;
  std::vector<int32_t> miss;
  miss.reserve((size_t)k);
  std::vector<int32_t>& tab = c->slot_sorted;
  tab.resize((size_t)k);
  std::vector<char> late((size_t)k, 0);  // fetched on demand by this layer
  size_t pi = 0;
  int64_t hits = 0;
  for (int64_t u = 0; u < k; ++u) {
    const int32_t j = c->sel_host[u];
    const int64_t cb = chunk_bytes(c, j);
    stv.bytes_gathered += cb;
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
      late[u] = 1;
      miss.push_back(j);
      stv.bytes_demand += cb;
    }
  }
  stv.hits = hits;
  stv.misses = (int64_t)miss.size();
  stv.wasted = (int64_t)P.size() - hits;
  const int64_t n_pred = (int64_t)P.size();
  // the attention's lists (pinned staging, one copy to the device): chunk
  // indices and slots of the kept chunks already in HBM, then of the misses,
  // each part in ascending chunk order.  The misses' indices are also the
  // demand copy's list.
  const int64_t n_early = k - (int64_t)miss.size();
  {
    int32_t* tabp = B.tab_host;
    int32_t* selp = B.dem_host;  // = tab_host + k (one staging block)
    int64_t e = 0, x = n_early;
    for (int64_t u = 0; u < k; ++u) {
      const int64_t at = late[u] ? x++ : e++;
      tabp[at] = tab[u];
      selp[at] = c->sel_host[u];
    }
  }

  // storage tier: the pool slots the misses move from; those not in the pool
  // get free slots and are read from the file below
  c->io_keys.clear();  // this layer's demand reads (none without misses)
  c->io_dst.clear();
  std::vector<int32_t> msrc, mdst;
  if (stored && !miss.empty()) {
    const size_t nm = miss.size();
    msrc.resize(nm);
    mdst.resize(nm);
    for (size_t i = 0; i < nm; ++i) {
      const int64_t x = key0 + miss[i];
      if (c->pool_of[x] < 0) {
        if (pool_take(c, x) < 0) CKV_FAIL(CKV_ESTATE, "chunk pool exhausted (internal)");
        c->io_keys.push_back(x);
        c->io_dst.push_back(c->pool + (int64_t)c->pool_of[x] * c->slot_bytes);
      }
      msrc[i] = c->pool_of[x];
      mdst[i] = (int32_t)(buf0 + n_pred + i);
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

  // The layer's own set is known: the rest of a Period is predicted exactly.
  // With intra-period prefetch the first layer of a Period queues the copies of
  // every later layer of the Period (behind its own demand copies) before its
  // attention goes out, so that the SubPeriod gate can wait for them.
  const bool pw = period_wide(c) && !reuse && c->period > 1;
  int32_t gate_layer = -1;
  auto period_prefetch = [&]() -> ckv_status {
    if (!pw) return CKV_OK;
    const int32_t last = std::min<int32_t>(first + c->period - 1, c->n_layers - 1);
    std::vector<int32_t> Pt;
    for (int32_t t = layer + 1; t <= last; ++t) {
      uncached(c, t, c->sel_host, k, Pt);
      ckv_status r = queue_prefetch(c, t % c->nbuf, t, c->host_layers[t], Pt, true,
                                    &stv.bytes_prefetch);
      if (r != CKV_OK) return r;
    }
    if (c->subperiod > 1) gate_layer = std::min<int32_t>(layer + c->subperiod - 1, last);
    return CKV_OK;
  };

  // demand copies into this layer's buffer (after the attention that last used
  // it; from the pool once its reads have landed), then the attention.  The
  // small index copies go first, so they never queue behind span copies.
  auto demand_and_attention = [&]() -> ckv_status {
    if (dem_ticket) {
      ckv_status w = store_wait(c->kv_store, dem_ticket);
      if (w != CKV_OK) return w;
    }
    if (c->inject_layer == layer) {  // test hook: the copy enqueue fails here
      c->inject_layer = -1;
      CKV_FAIL(CKV_EHIP, "injected host-to-HBM copy failure at layer %d", layer);
    }
    if (B.attn_rec) CKV_HIP(hipStreamWaitEvent(c->demand, B.ev_attn, 0));
    // slots then chunk indices: adjacent on the host and on the device
    CKV_HIP(hipMemcpyAsync(B.tab_dev, B.tab_host, (size_t)(2 * k) * sizeof(int32_t),
                           hipMemcpyHostToDevice, c->demand));
    CKV_HIP(hipEventRecord(c->ev_tab, c->demand));
    ckv_status r = CKV_OK;
    const int64_t nm = (int64_t)miss.size();
    // shares of the misses, each copied and then attended over on its own (from
    // the storage tier's pool one copy lands every share; the shares, and so
    // the roundings, stay those of the pinned-store path)
    const int parts = nm == 0 ? 0 : (int)std::min<int64_t>(ckv_ctx::kLateParts, nm);
    if (nm > 0 && stored) {
      // its staging guard, recorded after its own list copy, covers the lists above
      r = pool_copy(c, cur, 1, msrc.data(), mdst.data(), nm, c->demand);
      if (r != CKV_OK) return r;
      for (int i = 0; i < parts; ++i) CKV_HIP(hipEventRecord(c->ev_late[i], c->demand));
    } else {
      CKV_HIP(hipEventRecord(B.ev_gd, c->demand));
      B.gd = true;
      for (int i = 0; i < parts; ++i) {
        const int64_t b0 = attn_late_part_begin(nm, parts, i), b1 = attn_late_part_begin(nm, parts, i + 1);
        r = launch_copy_spans(la.store, B.dem_dev + n_early + b0, b1 - b0, n_pred + b0, B.slots,
                              c->slot_bytes, c->demand);
        if (r != CKV_OK) return r;
        CKV_HIP(hipEventRecord(c->ev_late[i], c->demand));
      }
    }
    CKV_HIP(hipEventRecord(c->ev_dem, c->demand));
    if ((r = period_prefetch()) != CKV_OK) return r;
    const bool parted = c->attn_splits > 0;
    CKV_HIP(hipStreamWaitEvent(st, parted ? c->ev_tab : c->ev_dem, 0));
    if (B.pref_pending) CKV_HIP(hipStreamWaitEvent(st, B.ev_pref, 0));
    B.pref_pending = false;
    if (gate_layer > layer) {  // SubPeriod gate: the Period's first layers are in HBM
      SlotBuf& Bg = c->buf[gate_layer % c->nbuf];
      CKV_HIP(hipStreamWaitEvent(st, Bg.ev_pref, 0));
    }
    if ((r = mark(4)) != CKV_OK) return r;
    ChunkSource src{c->arena, static_cast<char*>(c->arena) + span_elems * eb, 2 * span_elems,
                    B.tab_dev, 0, c->nbuf * spb + c->cache_slots};
    if (parted) {
      // the chunks already in HBM and the suffix while the misses are copied,
      // then each share of the misses once it has landed, then one merge of
      // every part's splits
      void* aw = ws + c->off_attn;
      int32_t done = 0, ns = 0;
      r = launch_attn_part(d, io->q, src, B.dem_dev, n_early, io->k_suffix, io->v_suffix, true, aw,
                           c->attn_splits, 0, &ns, st);
      if (r != CKV_OK) return r;
      done += ns;
      for (int i = 0; i < parts; ++i) {
        const int64_t b0 = attn_late_part_begin(nm, parts, i), b1 = attn_late_part_begin(nm, parts, i + 1);
        CKV_HIP(hipStreamWaitEvent(st, c->ev_late[i], 0));
        ChunkSource late = src;
        late.chunk_off = B.tab_dev + n_early + b0;
        r = launch_attn_part(d, io->q, late, B.dem_dev + n_early + b0, b1 - b0, io->k_suffix,
                             io->v_suffix, false, aw, c->attn_splits, done, &ns, st);
        if (r != CKV_OK) return r;
        done += ns;
      }
      CKV_HIP(hipStreamWaitEvent(st, c->ev_dem, 0));
      r = launch_attn_combine(d, aw, c->attn_splits, done, io->out, st);
    } else {
      r = launch_attn(d, io->q, src, B.dem_dev, k, io->k_suffix, io->v_suffix, io->out,
                      ws + c->off_attn, c->ws_attn, st);
    }
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
    if ((s = guard(B.ev_gf, B.gf)) != CKV_OK) return s;
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
    int32_t* fill = B.fill_host;
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

  const bool has_next = stored ? layer + 1 < c->store_layers : la.store_next != nullptr;
  if (stored && has_next) {
    // the next layer's prediction (P_{l+1} = S_l, less the chunks it will find
    // in the cache's HBM slots) joins the I/O threads' queue behind this
    // layer's demand reads and runs on while this layer attends and the next
    // one scores.  Layers last_ahead..: inside a Period with a SubPeriod of sp
    // layers, every layer up to sp - 1 ahead (their set is this one);
    // otherwise the next layer only (speculative across a Period boundary)
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
        stv.bytes_prefetch += chunk_bytes(c, j);
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
  if (stored && (s = demand_and_attention()) != CKV_OK) return s;

  if (nf > 0) {  // chunks entering the GPU tier, after the attention that read their slots
    CKV_HIP(hipMemcpyAsync(B.fill_dev, B.fill_host, (size_t)(2 * k) * sizeof(int32_t),
                           hipMemcpyHostToDevice, st));
    CKV_HIP(hipEventRecord(B.ev_gf, st));
    B.gf = true;
    s = launch_copy_slots(c->arena, B.fill_dev, c->arena, B.fill_dev + k, nf, c->slot_bytes, st);
    if (s != CKV_OK) return s;
    stv.bytes_cache_fill = nf * c->slot_bytes;
  }
  // after the cache fills too: they read this layer's buffer
  CKV_HIP(hipEventRecord(B.ev_attn, st));
  B.attn_rec = true;
  B.pred_layer = -1;  // consumed
  B.pred.clear();

  // the next layer's copy over the host link on the side stream, unless the
  // Period's prefetch has already queued it: P_{l+1} = S_l less the chunks the
  // next layer will find in the cache's HBM slots (after this layer's cache
  // decisions)
  if (!stored && has_next) {
    const int32_t t = layer + 1;
    const int bn = t % c->nbuf;
    if (c->buf[bn].pred_layer != t) {
      std::vector<int32_t> Pn;
      uncached(c, t, c->sel_host, k, Pn);
      s = queue_prefetch(c, bn, t, la.store_next, Pn, true, &stv.bytes_prefetch);
      if (s != CKV_OK) return s;
    }
  }
  c->prev_layer = layer;
  if (stats) *stats = stv;
  return CKV_OK;
}

}  // namespace
