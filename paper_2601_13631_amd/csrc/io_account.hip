// io_account.hip -- read accounting of a chunk selection (host code).
// Sec. 4.2: a ContiguousChunk store reads exactly the selected chunks.
// Sec. 3, Motivation 1: a store cut into fixed coarse blocks reads every block
// that holds a needed token.  One pass over the ascending selection: each
// chunk's token span [t0, t1) covers blocks t0/b .. (t1-1)/b, of which those
// past the last block already counted are new.

#include "ckv_internal.h"

using namespace ckv;

extern "C" ckv_status ckv_io_account(int64_t n, int32_t c, const int32_t* sel_idx, int64_t k,
                                     int32_t block_tokens, ckv_io_counts* out) {
  clear_error();
  if (n < 1 || c < 1 || block_tokens < 1)
    CKV_FAIL(CKV_EINVAL, "n, c and block_tokens must be >= 1 (got %lld, %d, %d)", (long long)n, c,
             block_tokens);
  if (!out || (k > 0 && !sel_idx)) CKV_FAIL(CKV_EINVAL, "NULL pointer argument");
  const int64_t m = (n + c - 1) / c;
  if (k < 0 || k > m) CKV_FAIL(CKV_EINVAL, "k must be in [0, %lld] (got %lld)", (long long)m, (long long)k);
  for (int64_t u = 0; u < k; ++u) {
    if (sel_idx[u] < 0 || sel_idx[u] >= m)
      CKV_FAIL(CKV_EINVAL, "sel_idx[%lld] = %d outside [0, %lld)", (long long)u, sel_idx[u], (long long)m);
    if (u > 0 && sel_idx[u] <= sel_idx[u - 1])
      CKV_FAIL(CKV_EINVAL, "sel_idx must be strictly ascending (position %lld)", (long long)u);
  }
  const int64_t b = block_tokens;
  ckv_io_counts r = {0, 0, 0, 0};
  int64_t last_block = -1;
  for (int64_t u = 0; u < k; ++u) {
    const int64_t j = sel_idx[u];
    const int64_t t0 = j * c, t1 = std::min<int64_t>(t0 + c, n);
    r.tokens_selected += t1 - t0;
    if (u == 0 || sel_idx[u - 1] != j - 1) r.runs++;
    const int64_t b0 = std::max(t0 / b, last_block + 1), b1 = (t1 - 1) / b;
    if (b0 <= b1) {
      r.blocks += b1 - b0 + 1;
      r.tokens_block += std::min(n, (b1 + 1) * b) - b0 * b;  // only the prefix's last block is short
      last_block = b1;
    }
  }
  *out = r;
  return CKV_OK;
}
