// Host-code driver for sanitizer builds: exercises the attention-guided cache (random request streams, every query call, a refused request) and the read accounting (random selections) through the C ABI.
// Built and run by tests/test_sanitizers.py with -fsanitize=address or thread on the host side only.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>
#include <cstring>
#include "ckv.h"
int main() {
  std::mt19937_64 rng(7);
  for (int trial = 0; trial < 200; ++trial) {
    int64_t n_keys = 1 + rng() % 500, g = rng() % 60, c = rng() % 60;
    ckv_cache* cache = nullptr;
    if (ckv_cache_create(n_keys, g, c, (int)(rng() % 2), &cache) != CKV_OK) { printf("create fail\n"); return 1; }
    std::vector<int64_t> keys; std::vector<double> A; std::vector<int8_t> where;
    for (int r = 0; r < 300; ++r) {
      int64_t cnt = rng() % std::min<int64_t>(n_keys, 40);
      std::vector<char> used(n_keys, 0);
      keys.clear(); A.clear();
      while ((int64_t)keys.size() < cnt) { int64_t x = rng() % n_keys; if (!used[x]) { used[x] = 1; keys.push_back(x); A.push_back((rng() % 100) * 0.25); } }
      where.assign(cnt, 0);
      ckv_cache_counts counts;
      if (ckv_cache_access(cache, keys.data(), A.data(), cnt, where.data(), &counts) != CKV_OK) { printf("access fail\n"); return 1; }
      if (r % 50 == 0) {
        std::vector<int64_t> res(n_keys); int64_t n = 0;
        ckv_cache_resident(cache, CKV_TIER_GPU, res.data(), n_keys, &n);
        ckv_cache_resident(cache, CKV_TIER_CPU, res.data(), n_keys, &n);
        std::vector<double> I(n_keys); std::vector<int64_t> F(n_keys); std::vector<int8_t> T(n_keys);
        ckv_cache_state(cache, I.data(), F.data(), T.data());
      }
    }
    // invalid requests
    int64_t dup[2] = {0, 0}; double a2[2] = {1, 1};
    if (n_keys >= 1 && ckv_cache_access(cache, dup, a2, 2, nullptr, nullptr) != CKV_EINVAL) { printf("dup not refused\n"); return 1; }
    ckv_cache_destroy(cache);
  }
  for (int trial = 0; trial < 2000; ++trial) {
    int64_t n = 1 + rng() % 5000; int32_t cc = 1 + rng() % 70, b = 1 + rng() % 130;
    int64_t m = (n + cc - 1) / cc;
    std::vector<int32_t> sel;
    for (int64_t j = 0; j < m; ++j) if (rng() % 3 == 0) sel.push_back((int32_t)j);
    ckv_io_counts out;
    if (ckv_io_account(n, cc, sel.data(), (int64_t)sel.size(), b, &out) != CKV_OK) { printf("io fail\n"); return 1; }
  }
  printf("cache and read-accounting drive ok\n");
  return 0;
}
