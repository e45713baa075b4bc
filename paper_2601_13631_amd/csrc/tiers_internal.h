// tiers_internal.h -- internals shared by the layer context and the memory
// tiers it drives: HBM slot copies, the storage tier and the attention-guided
// cache (libckv, gfx950 only).
#pragma once

#include <vector>

#include "ckv_internal.h"

namespace ckv {

// Copies whole spans of span_bytes each: span src_slots[i] of src to span
// dst_slots[i] of dst, for i < count; both lists are device arrays.  For
// device-to-device moves and moves out of the pinned chunk pool (a wider grid
// than launch_copy_spans).
ckv_status launch_copy_slots(const void* src, const int32_t* src_slots, void* dst,
                             const int32_t* dst_slots, int64_t count, int64_t span_bytes,
                             hipStream_t st);

// ---- storage tier, as a layer context drives it ------------------------------
int64_t store_keys(const ckv_store* s);
int64_t store_span_bytes(const ckv_store* s);
bool store_direct(const ckv_store* s);
// Queues reads of spans keys[u] into dst[u] (host memory) for the I/O threads;
// *ticket names the request for store_wait.
ckv_status store_submit(ckv_store* s, const int64_t* keys, int64_t count, char* const* dst,
                        int64_t* ticket);
// Blocks until every read of the ticket has landed (CKV_EHIP on a read error).
ckv_status store_wait(ckv_store* s, int64_t ticket);

// ---- attention-guided cache, as a layer context drives it ------------------
int64_t cache_keys(const ckv_cache* c);
int64_t cache_gpu_slots(const ckv_cache* c);
int64_t cache_cpu_slots(const ckv_cache* c);
int64_t cache_gpu_size(const ckv_cache* c);
int8_t cache_tier(const ckv_cache* c, int64_t key);
// Starts (or stops) logging the keys that the cascade displaces from the GPU
// tier and the keys it sends out of memory.
void cache_log_gpu_evictions(ckv_cache* c, bool on);
// Moves the logged GPU-tier displacements into out (replacing its contents).
void cache_take_gpu_evictions(ckv_cache* c, std::vector<int64_t>& out);
// Moves the logged keys that left memory (or were not kept) into out.
void cache_take_drops(ckv_cache* c, std::vector<int64_t>& out);

}  // namespace ckv
