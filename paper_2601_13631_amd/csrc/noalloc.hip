// noalloc.hip -- the HBM-resident layer step with no allocation of any kind,
// for callers that cannot allocate device memory (code under HIP graph
// capture, tight serving loops, harnesses that forbid it).
//
// Its scratch (the scoring workspace, the attention's split partials and, when
// the caller passes no output for them, the chunk scores and the kept set) is
// one file-scope device array of kScratchBytes.  Host code never uses the
// array's name as an address: on each device's first call the device address
// of that device's copy is looked up once (hipGetSymbolAddress) and kept, and
// every kernel gets that pointer.  The same kernels and the same scratch
// layout as a layer-step context run, so results are bit-identical to
// ckv_reprefill_layer on an HBM-resident context.  Calls on one device share
// the array: calls that overlap in time on one device race.

#include <mutex>

#include "ckv_internal.h"

namespace {

constexpr size_t kScratchBytes = size_t(64) << 20;
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

// The device address of the current device's copy of `scratch`.
ckv_status scratch_on_current_device(void** out) {
  int dev = -1;
  CKV_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices)
    CKV_FAIL(CKV_EUNSUPPORTED, "device %d is beyond the %d devices this entry point serves", dev,
             kMaxDevices);
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    CKV_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) CKV_FAIL(CKV_EHIP, "no device address for the scratch array");
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return CKV_OK;
}

}  // namespace

using namespace ckv;

extern "C" {

ckv_status ckv_reprefill_layer_noalloc(const ckv_dims* dims, double keep_ratio, const void* q,
                                       const void* k_prefix, const void* v_prefix,
                                       const void* k_suffix, const void* v_suffix, void* out,
                                       double* chunk_scores, int32_t* sel_idx, void* stream) {
  clear_error();
  {
    ckv_status s = check_dims(dims);
    if (s != CKV_OK) return s;
  }
  if (!(keep_ratio > 0.0 && keep_ratio <= 1.0)) CKV_FAIL(CKV_EINVAL, "keep_ratio must be in (0, 1]");
  if (!q || !k_prefix || !v_prefix || !k_suffix || !v_suffix || !out)
    CKV_FAIL(CKV_EINVAL, "NULL tensor argument");
  if (!aligned16(q) || !aligned16(k_prefix) || !aligned16(v_prefix) || !aligned16(k_suffix) ||
      !aligned16(v_suffix) || !aligned16(out) || !aligned16(chunk_scores) || !aligned16(sel_idx))
    CKV_FAIL(CKV_EINVAL, "tensors must be 16-byte aligned");
  const int64_t m = ckv_num_chunks(dims->n_prefix, dims->chunk_size);
  const int64_t k = ckv_num_keep(m, keep_ratio);
  const size_t ws_score = make_score_plan(dims).bytes;
  if (ws_score == 0) CKV_FAIL(CKV_EUNSUPPORTED, "shape too large for the scoring decomposition");
  const size_t ws_attn = make_attn_plan(dims, k).bytes;
  // the layout of a layer-step context: scoring and attention scratch at the
  // front (used one after the other on one stream), then scores, then the set
  size_t off = align_up(std::max(ws_score, ws_attn), 256);
  const size_t off_scores = off;
  if (!chunk_scores) off = align_up(off + (size_t)m * sizeof(double), 256);
  const size_t off_sel = off;
  if (!sel_idx) off = align_up(off + (size_t)k * sizeof(int32_t), 256);
  if (off > kScratchBytes)
    CKV_FAIL(CKV_EINVAL, "this shape needs %zu bytes of scratch, above the %zu-byte maximum", off,
             kScratchBytes);
  void* base = nullptr;
  {
    ckv_status s = scratch_on_current_device(&base);
    if (s != CKV_OK) return s;
  }
  char* ws = static_cast<char*>(base);
  double* scores = chunk_scores ? chunk_scores : reinterpret_cast<double*>(ws + off_scores);
  int32_t* sel = sel_idx ? sel_idx : reinterpret_cast<int32_t*>(ws + off_sel);
  hipStream_t st = (hipStream_t)stream;
  ckv_status s = launch_score(dims, q, k_prefix, scores, ws, ws_score, st);
  if (s != CKV_OK) return s;
  s = launch_select(scores, m, k, sel, nullptr, 0, st);
  if (s != CKV_OK) return s;
  const int64_t span_elems = (int64_t)dims->chunk_size * dims->n_kv_heads * dims->head_dim;
  ChunkSource src{k_prefix, v_prefix, span_elems, nullptr, 1, m};
  return launch_attn(dims, q, src, sel, k, k_suffix, v_suffix, out, ws, ws_attn, st);
}

}  // extern "C"
