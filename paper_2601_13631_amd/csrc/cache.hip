// cache.hip -- attention-guided cache management (Sec. 4.5, Eq. 2), host code.
// Per key: I (sum of the attention scores of the requests that used it), F (that
// number of requests; with CKV_CACHE_LOADS the number of those uses that loaded
// the chunk into GPU or CPU memory, i.e. found it outside the GPU tier), the
// time of its latest use, and S = I*F (or F alone for the frequency-only
// policy).  The GPU and CPU tiers are indexed binary
// min-heaps on (S, latest use), so the weakest entry is at the root and any
// entry can be taken out when its key is used again.  A key's S changes only
// when it is used, and it is out of its heap at that moment, so the heaps stay
// ordered without sift-ups on score changes.

#include <cstring>
#include <new>
#include <vector>

#include "tiers_internal.h"

struct ckv_cache {
  int64_t n_keys = 0;
  int64_t slots[3] = {0, 0, 0};  // indexed by tier: [CKV_TIER_CPU], [CKV_TIER_GPU]
  int32_t policy = CKV_CACHE_ATTENTION;
  std::vector<double> I, S;
  std::vector<int64_t> F, last, pos, seen;
  std::vector<int8_t> tier;
  std::vector<int64_t> heap[3];
  int64_t clock = 0, call = 0;
  ckv_cache_counts counts = {0, 0, 0, 0, 0};
  // keys displaced from the GPU tier since the last drain (kept only while a
  // layer context holds the GPU tier's chunks in HBM)
  bool log_gpu_evictions = false;
  std::vector<int64_t> gpu_evicted;
  std::vector<int64_t> dropped_log;  // keys the cascade sent out of memory (same switch)
};

namespace {

// x leaves before y: lower score, then older latest use
inline bool weaker(const ckv_cache& c, int64_t x, int64_t y) {
  if (c.S[x] != c.S[y]) return c.S[x] < c.S[y];
  return c.last[x] < c.last[y];
}

void sift_up(ckv_cache& c, std::vector<int64_t>& h, int64_t i) {
  const int64_t x = h[i];
  while (i > 0) {
    const int64_t p = (i - 1) / 2;
    if (!weaker(c, x, h[p])) break;
    h[i] = h[p];
    c.pos[h[i]] = i;
    i = p;
  }
  h[i] = x;
  c.pos[x] = i;
}

void sift_down(ckv_cache& c, std::vector<int64_t>& h, int64_t i) {
  const int64_t n = (int64_t)h.size(), x = h[i];
  for (;;) {
    int64_t ch = 2 * i + 1;
    if (ch >= n) break;
    if (ch + 1 < n && weaker(c, h[ch + 1], h[ch])) ++ch;
    if (!weaker(c, h[ch], x)) break;
    h[i] = h[ch];
    c.pos[h[i]] = i;
    i = ch;
  }
  h[i] = x;
  c.pos[x] = i;
}

void heap_push(ckv_cache& c, int t, int64_t x) {
  std::vector<int64_t>& h = c.heap[t];
  h.push_back(x);
  c.tier[x] = (int8_t)t;
  sift_up(c, h, (int64_t)h.size() - 1);
}

void heap_erase(ckv_cache& c, int t, int64_t x) {
  std::vector<int64_t>& h = c.heap[t];
  const int64_t i = c.pos[x], tail = h.back();
  h.pop_back();
  c.tier[x] = CKV_TIER_NONE;
  if (tail == x) return;
  h[i] = tail;
  c.pos[tail] = i;
  sift_up(c, h, i);
  sift_down(c, h, c.pos[tail]);
}

// x joins tier t if it has room or x outranks its weakest entry, which is then
// returned (-1 if none left); x itself is returned when it is not taken.
int64_t admit(ckv_cache& c, int t, int64_t x) {
  std::vector<int64_t>& h = c.heap[t];
  if ((int64_t)h.size() < c.slots[t]) {
    heap_push(c, t, x);
    return -1;
  }
  if (h.empty() || !weaker(c, h[0], x)) return x;
  const int64_t y = h[0];
  heap_erase(c, t, y);
  heap_push(c, t, x);
  return y;
}

void place(ckv_cache& c, int64_t x) {
  int64_t out = admit(c, CKV_TIER_GPU, x);
  if (out < 0) return;
  const bool demoting = out != x;  // a GPU-tier entry goes down
  if (demoting && c.log_gpu_evictions) c.gpu_evicted.push_back(out);
  const int64_t left = admit(c, CKV_TIER_CPU, out);
  if (demoting && left != out) c.counts.demoted++;
  if (left >= 0) {
    c.counts.dropped++;
    if (c.log_gpu_evictions) c.dropped_log.push_back(left);
  }
}

}  // namespace

namespace ckv {

int64_t cache_keys(const ckv_cache* c) { return c->n_keys; }
int64_t cache_gpu_slots(const ckv_cache* c) { return c->slots[CKV_TIER_GPU]; }
int64_t cache_gpu_size(const ckv_cache* c) { return (int64_t)c->heap[CKV_TIER_GPU].size(); }
int8_t cache_tier(const ckv_cache* c, int64_t key) { return c->tier[key]; }

void cache_log_gpu_evictions(ckv_cache* c, bool on) {
  c->log_gpu_evictions = on;
  c->gpu_evicted.clear();
  c->dropped_log.clear();
}

void cache_take_drops(ckv_cache* c, std::vector<int64_t>& out) {
  out.swap(c->dropped_log);
  c->dropped_log.clear();
}

int64_t cache_cpu_slots(const ckv_cache* c) { return c->slots[CKV_TIER_CPU]; }

void cache_take_gpu_evictions(ckv_cache* c, std::vector<int64_t>& out) {
  out.swap(c->gpu_evicted);
  c->gpu_evicted.clear();
}

}  // namespace ckv

using namespace ckv;

extern "C" {

ckv_status ckv_cache_create(int64_t n_keys, int64_t gpu_slots, int64_t cpu_slots, int32_t policy,
                            ckv_cache** out) {
  clear_error();
  if (!out) CKV_FAIL(CKV_EINVAL, "out is NULL");
  *out = nullptr;
  if (n_keys < 1 || gpu_slots < 0 || cpu_slots < 0)
    CKV_FAIL(CKV_EINVAL, "n_keys must be >= 1 and slot counts >= 0");
  if (policy != CKV_CACHE_ATTENTION && policy != CKV_CACHE_LFU && policy != CKV_CACHE_LOADS)
    CKV_FAIL(CKV_EINVAL, "unknown cache policy %d", policy);
  ckv_cache* c = new (std::nothrow) ckv_cache;
  if (!c) CKV_FAIL(CKV_ENOMEM, "cache allocation failed");
  try {
    c->n_keys = n_keys;
    c->slots[CKV_TIER_GPU] = gpu_slots;
    c->slots[CKV_TIER_CPU] = cpu_slots;
    c->policy = policy;
    c->I.assign(n_keys, 0.0);
    c->S.assign(n_keys, 0.0);
    c->F.assign(n_keys, 0);
    c->last.assign(n_keys, 0);
    c->pos.assign(n_keys, -1);
    c->seen.assign(n_keys, 0);
    c->tier.assign(n_keys, CKV_TIER_NONE);
    c->heap[CKV_TIER_GPU].reserve(std::min(gpu_slots, n_keys));
    c->heap[CKV_TIER_CPU].reserve(std::min(cpu_slots, n_keys));
  } catch (...) {
    delete c;
    CKV_FAIL(CKV_ENOMEM, "cache allocation failed (%lld keys)", (long long)n_keys);
  }
  *out = c;
  return CKV_OK;
}

ckv_status ckv_cache_destroy(ckv_cache* cache) {
  clear_error();
  delete cache;
  return CKV_OK;
}

ckv_status ckv_cache_access(ckv_cache* cache, const int64_t* keys, const double* scores,
                            int64_t count, int8_t* tier_before, ckv_cache_counts* counts) {
  clear_error();
  if (!cache) CKV_FAIL(CKV_EINVAL, "cache is NULL");
  if (count < 0 || (count > 0 && (!keys || !scores)))
    CKV_FAIL(CKV_EINVAL, "keys and scores required for count %lld", (long long)count);
  ckv_cache& c = *cache;
  const int64_t call = ++c.call;  // marks keys seen in this call
  for (int64_t u = 0; u < count; ++u) {
    const int64_t x = keys[u];
    if (x < 0 || x >= c.n_keys) {
      CKV_FAIL(CKV_EINVAL, "keys[%lld] = %lld outside [0, %lld)", (long long)u, (long long)x,
               (long long)c.n_keys);
    }
    if (!(scores[u] >= 0.0) || std::isinf(scores[u]))
      CKV_FAIL(CKV_EINVAL, "scores[%lld] must be finite and >= 0", (long long)u);
    if (c.seen[x] == call) CKV_FAIL(CKV_EINVAL, "key %lld repeated in one request", (long long)x);
    c.seen[x] = call;
  }
  for (int64_t u = 0; u < count; ++u) {
    const int64_t x = keys[u];
    const int8_t was = c.tier[x];
    if (tier_before) tier_before[u] = was;
    if (was == CKV_TIER_GPU) c.counts.hits_gpu++;
    else if (was == CKV_TIER_CPU) c.counts.hits_cpu++;
    else c.counts.misses++;
    if (was != CKV_TIER_NONE) heap_erase(c, was, x);
    c.I[x] += scores[u];
    if (c.policy != CKV_CACHE_LOADS || was != CKV_TIER_GPU) c.F[x] += 1;  // a use, or a load
    c.last[x] = ++c.clock;
    c.S[x] = c.policy == CKV_CACHE_LFU ? (double)c.F[x] : c.I[x] * (double)c.F[x];
    place(c, x);
  }
  if (counts) *counts = c.counts;
  return CKV_OK;
}

ckv_status ckv_cache_lookup(const ckv_cache* cache, const int64_t* keys, int64_t count,
                            int8_t* tier) {
  clear_error();
  if (!cache || count < 0 || (count > 0 && (!keys || !tier)))
    CKV_FAIL(CKV_EINVAL, "NULL pointer or negative count");
  for (int64_t u = 0; u < count; ++u)
    if (keys[u] < 0 || keys[u] >= cache->n_keys)
      CKV_FAIL(CKV_EINVAL, "keys[%lld] out of range", (long long)u);
  for (int64_t u = 0; u < count; ++u) tier[u] = cache->tier[keys[u]];
  return CKV_OK;
}

ckv_status ckv_cache_state(const ckv_cache* cache, double* importance, int64_t* frequency,
                           int8_t* tier) {
  clear_error();
  if (!cache) CKV_FAIL(CKV_EINVAL, "cache is NULL");
  const size_t n = (size_t)cache->n_keys;
  if (importance) std::memcpy(importance, cache->I.data(), n * sizeof(double));
  if (frequency) std::memcpy(frequency, cache->F.data(), n * sizeof(int64_t));
  if (tier) std::memcpy(tier, cache->tier.data(), n);
  return CKV_OK;
}

ckv_status ckv_cache_resident(const ckv_cache* cache, int32_t tier, int64_t* keys,
                              int64_t capacity, int64_t* n) {
  clear_error();
  if (!cache || !n || (tier != CKV_TIER_CPU && tier != CKV_TIER_GPU))
    CKV_FAIL(CKV_EINVAL, "NULL pointer or tier not CPU/GPU");
  const std::vector<int64_t>& h = cache->heap[tier];
  *n = (int64_t)h.size();
  if ((int64_t)h.size() > capacity || (!h.empty() && !keys))
    CKV_FAIL(CKV_EINVAL, "tier holds %lld keys, capacity %lld", (long long)h.size(),
             (long long)capacity);
  int64_t w = 0;
  for (int64_t x = 0; x < cache->n_keys && w < (int64_t)h.size(); ++x)
    if (cache->tier[x] == tier) keys[w++] = x;
  return CKV_OK;
}

}  // extern "C"
