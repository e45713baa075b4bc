// api.hip -- C ABI of libckv: argument validation and dispatch to the kernels.
// Every entry point validates before it enqueues anything; no C++ exception
// leaves this file.

#include <cstdarg>
#include <cstring>
#include <new>

#include "ckv_internal.h"

namespace ckv {

namespace {
thread_local char g_err[512] = "";
}

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
}
void clear_error() { g_err[0] = 0; }

ckv_status check_dims(const ckv_dims* d) {
  if (!d) CKV_FAIL(CKV_EINVAL, "dims is NULL");
  if (d->n_prefix < 1) CKV_FAIL(CKV_EINVAL, "n_prefix must be >= 1 (got %lld)", (long long)d->n_prefix);
  if (d->n_suffix < 1) CKV_FAIL(CKV_EINVAL, "n_suffix must be >= 1 (got %d)", d->n_suffix);
  if (d->n_q_heads < 1 || d->n_kv_heads < 1 || d->n_q_heads % d->n_kv_heads)
    CKV_FAIL(CKV_EINVAL, "n_q_heads (%d) must be a positive multiple of n_kv_heads (%d)",
             d->n_q_heads, d->n_kv_heads);
  if (d->chunk_size < 1) CKV_FAIL(CKV_EINVAL, "chunk_size must be >= 1 (got %d)", d->chunk_size);
  if (!(d->sm_scale >= 0.f) || std::isinf(d->sm_scale))
    CKV_FAIL(CKV_EINVAL, "sm_scale must be finite and >= 0");
  if (d->dtype != CKV_DTYPE_F32 && d->dtype != CKV_DTYPE_BF16)
    CKV_FAIL(CKV_EINVAL, "unknown dtype %d", d->dtype);
  if (d->head_dim < 1) CKV_FAIL(CKV_EINVAL, "head_dim must be >= 1");
  if (d->dtype == CKV_DTYPE_BF16 && d->head_dim != 64 && d->head_dim != 128)
    CKV_FAIL(CKV_EUNSUPPORTED, "bf16 supports head_dim 64 or 128 (got %d)", d->head_dim);
  if (d->dtype == CKV_DTYPE_F32 && d->head_dim != 64)
    CKV_FAIL(CKV_EUNSUPPORTED, "fp32 supports head_dim 64 (got %d)", d->head_dim);
  const int c = d->chunk_size;
  if (!(c == 4 || c == 8 || c == 16 || c % 32 == 0))
    CKV_FAIL(CKV_EUNSUPPORTED, "chunk_size must be 4, 8, 16 or a multiple of 32 (got %d)", c);
  const int64_t rows = (int64_t)(d->n_q_heads / d->n_kv_heads) * d->n_suffix;
  if (rows > (1 << 24) || d->n_prefix > (int64_t(1) << 30))
    CKV_FAIL(CKV_EUNSUPPORTED, "shape too large");
  return CKV_OK;
}

}  // namespace ckv

using namespace ckv;

#define CKV_REQUIRE(cond, ...)                      \
  do {                                              \
    if (!(cond)) CKV_FAIL(CKV_EINVAL, __VA_ARGS__); \
  } while (0)

#define CKV_CHECK(expr)            \
  do {                             \
    ckv_status s_ = (expr);        \
    if (s_ != CKV_OK) return s_;   \
  } while (0)

extern "C" {

const char* ckv_last_error(void) { return g_err; }

const char* ckv_version(void) { return "libckv 0.1 (gfx950)"; }

int64_t ckv_num_chunks(int64_t n, int32_t c) {
  if (n < 0 || c < 1) return -1;
  return (n + c - 1) / c;
}

int64_t ckv_num_keep(int64_t m, double r) {
  if (!(r > 0.0 && r <= 1.0) || m < 0) return -1;
  if (m == 0) return 0;
  int64_t k = (int64_t)std::ceil(r * (double)m - 1e-9);
  return std::max<int64_t>(1, std::min<int64_t>(k, m));
}

size_t ckv_score_workspace_bytes(const ckv_dims* dims) {
  if (check_dims(dims) != CKV_OK) return 0;
  return make_score_plan(dims).bytes;
}

ckv_status ckv_score_chunks(const ckv_dims* dims, const void* q, const void* k_prefix,
                            double* chunk_scores, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  CKV_CHECK(check_dims(dims));
  CKV_REQUIRE(q && k_prefix && chunk_scores && ws, "NULL pointer argument");
  CKV_REQUIRE(aligned16(q) && aligned16(k_prefix) && aligned16(chunk_scores) && aligned16(ws),
              "pointers must be 16-byte aligned");
  const size_t need = make_score_plan(dims).bytes;
  CKV_REQUIRE(ws_bytes >= need, "workspace too small: %zu < %zu", ws_bytes, need);
  return launch_score(dims, q, k_prefix, chunk_scores, ws, ws_bytes, (hipStream_t)stream);
}

size_t ckv_select_workspace_bytes(int64_t m) { return select_ws_bytes(m); }

ckv_status ckv_select_topk_chunks(const double* chunk_scores, int64_t m, int64_t k,
                                  int32_t* sel_idx, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  CKV_REQUIRE(chunk_scores && sel_idx, "NULL pointer argument");
  CKV_REQUIRE(m >= 1 && m <= INT32_MAX, "m must be in [1, 2^31-1] (got %lld)", (long long)m);
  CKV_REQUIRE(k >= 1 && k <= m, "k must be in [1, m] (got k=%lld, m=%lld)", (long long)k, (long long)m);
  CKV_REQUIRE(ws_bytes >= select_ws_bytes(m), "workspace too small");
  return launch_select(chunk_scores, m, k, sel_idx, ws, ws_bytes, (hipStream_t)stream);
}

ckv_status ckv_gather_chunks(const ckv_dims* dims, const void* k_src, const void* v_src,
                             const int32_t* sel_idx, int64_t k, void* k_sel, void* v_sel,
                             void* stream) {
  clear_error();
  CKV_CHECK(check_dims(dims));
  const int64_t m = ckv_num_chunks(dims->n_prefix, dims->chunk_size);
  CKV_REQUIRE(k >= 0 && k <= m, "k must be in [0, m] (got %lld)", (long long)k);
  if (k == 0) return CKV_OK;
  CKV_REQUIRE(k_src && v_src && sel_idx && k_sel && v_sel, "NULL pointer argument");
  CKV_REQUIRE(aligned16(k_src) && aligned16(v_src) && aligned16(k_sel) && aligned16(v_sel),
              "pointers must be 16-byte aligned");
  const int64_t row_bytes = (int64_t)dims->n_kv_heads * dims->head_dim * elem_bytes(dims->dtype);
  CKV_REQUIRE(row_bytes % 16 == 0, "Hkv*d*elem_bytes must be a multiple of 16");
  const void* ks = device_view(k_src);
  const void* vs = device_view(v_src);
  CKV_REQUIRE(ks && vs, "k_src/v_src must be device memory or pinned host memory");
  return launch_gather(dims, ks, vs, sel_idx, k, k_sel, v_sel, (hipStream_t)stream);
}

size_t ckv_attn_workspace_bytes(const ckv_dims* dims, int64_t k) {
  if (check_dims(dims) != CKV_OK || k < 0) return 0;
  return make_attn_plan(dims, k).bytes;
}

ckv_status ckv_sparse_prefill_attn(const ckv_dims* dims, const void* q, const void* k_sel,
                                   const void* v_sel, const int32_t* sel_idx, int64_t k,
                                   const void* k_suffix, const void* v_suffix, void* out,
                                   void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  CKV_CHECK(check_dims(dims));
  const int64_t m = ckv_num_chunks(dims->n_prefix, dims->chunk_size);
  CKV_REQUIRE(k >= 0 && k <= m, "k must be in [0, m] (got %lld)", (long long)k);
  CKV_REQUIRE(q && k_suffix && v_suffix && out, "NULL pointer argument");
  CKV_REQUIRE(k == 0 || (k_sel && v_sel && sel_idx), "NULL chunk argument with k > 0");
  CKV_REQUIRE(aligned16(q) && aligned16(k_suffix) && aligned16(v_suffix) && aligned16(out) &&
                  aligned16(k_sel) && aligned16(v_sel),
              "pointers must be 16-byte aligned");
  const size_t need = make_attn_plan(dims, k).bytes;
  CKV_REQUIRE(need == 0 || (ws && ws_bytes >= need), "workspace too small: %zu < %zu", ws_bytes, need);
  ChunkSource src{k_sel, v_sel, (int64_t)dims->chunk_size * dims->n_kv_heads * dims->head_dim,
                  nullptr, 0, k};
  return launch_attn(dims, q, src, sel_idx, k, k_suffix, v_suffix, out, ws, ws_bytes,
                     (hipStream_t)stream);
}

}  // extern "C"
