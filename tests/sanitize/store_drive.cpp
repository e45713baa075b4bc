// Host-code driver for sanitizer builds: exercises the storage tier's reader (random key lists with runs, buffered and O_DIRECT, misaligned destinations, a refused key) against the file's bytes through the C ABI.
// Built and run by tests/test_sanitizers.py with -fsanitize=address or thread on the host side only.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>
#include <cstring>
#include "ckv.h"
int main() {
  const int64_t span = 8192, n = 600;
  std::vector<unsigned char> data(span * n);
  std::mt19937_64 rng(3);
  for (auto& x : data) x = (unsigned char)rng();
  FILE* f = fopen("store.bin", "wb"); fwrite(data.data(), 1, data.size(), f); fclose(f);
  for (int flags = 0; flags < 2; ++flags) {
    ckv_store* st = nullptr;
    if (ckv_store_open("store.bin", n, span, 7, flags, &st) != CKV_OK) { printf("open fail %s\n", ckv_last_error()); return 1; }
    for (int t = 0; t < 300; ++t) {
      int64_t cnt = rng() % 40;
      std::vector<int64_t> keys(cnt);
      int64_t k0 = rng() % n;
      for (int64_t i = 0; i < cnt; ++i) keys[i] = (rng() % 3 == 0) ? (k0 + i) % n : rng() % n;
      std::vector<unsigned char> out(cnt * span + 1);
      if (ckv_store_read(st, keys.data(), cnt, out.data() + (t % 2)) != CKV_OK) { printf("read fail %s\n", ckv_last_error()); return 1; }
      for (int64_t i = 0; i < cnt; ++i)
        if (memcmp(out.data() + (t % 2) + i * span, data.data() + keys[i] * span, span)) { printf("mismatch\n"); return 1; }
    }
    int64_t bad = n;
    if (ckv_store_read(st, &bad, 1, data.data()) != CKV_EINVAL) { printf("bad key accepted\n"); return 1; }
    ckv_store_close(st);
  }
  remove("store.bin");
  printf("store drive ok\n");
  return 0;
}
