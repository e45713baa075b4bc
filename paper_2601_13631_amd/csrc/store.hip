// store.hip -- the storage tier (Sec. 4.3.2 and Sec. 4.5: prefix KV on SSD,
// loaded by I/O threads into host memory, then moved to the GPU).  Host code.
//
// The store is one file of n_keys spans of span_bytes each; span `key` sits at
// byte offset key * span_bytes (for a layer context, key = layer * m + chunk
// and each span is one chunk's K rows then V rows, the host-resident layout).
// A read request is a list of (key, destination) pairs; runs of consecutive
// keys with consecutive destinations become one pread, cut into pieces of at
// most kPieceBytes, and a pool of I/O threads takes the pieces in order.  With
// CKV_STORE_DIRECT the file is opened with O_DIRECT (no page cache), which
// needs span_bytes to be a multiple of 4096; each I/O thread then reads into
// its own aligned bounce buffer and copies to the destination (direct reads
// into pinned device-mapped memory are refused by the kernel).

#include <fcntl.h>
#include <stdlib.h>
#include <unistd.h>

#include <cerrno>
#include <condition_variable>
#include <cstring>
#include <deque>
#include <mutex>
#include <new>
#include <thread>
#include <vector>

#include "tiers_internal.h"

namespace {

constexpr int64_t kPieceBytes = 4 << 20;
constexpr int64_t kDirectAlign = 4096;

struct ReadJob {
  int64_t offset, bytes;
  char* dst;
  int64_t ticket;
};

}  // namespace

struct ckv_store {
  int fd = -1;
  int64_t n_keys = 0, span_bytes = 0;
  bool direct = false;
  std::vector<std::thread> threads;
  std::mutex mu;
  std::condition_variable cv_work, cv_done;
  std::deque<ReadJob> queue;
  int64_t next_ticket = 1;
  std::vector<int64_t> pending;  // pieces left per ticket, indexed ticket % kTickets
  std::vector<int> failed;       // errno of the ticket's first failed piece
  bool stop = false;
  static constexpr int kTickets = 64;
};

namespace ckv {
namespace {

void io_worker(ckv_store* s) {
  char* bounce = nullptr;  // direct reads land here first
  if (s->direct && posix_memalign(reinterpret_cast<void**>(&bounce), kDirectAlign, kPieceBytes))
    bounce = nullptr;
  for (;;) {
    ReadJob j;
    {
      std::unique_lock<std::mutex> lk(s->mu);
      s->cv_work.wait(lk, [&] { return s->stop || !s->queue.empty(); });
      if (s->queue.empty()) {  // stop requested and nothing left
        free(bounce);
        return;
      }
      j = s->queue.front();
      s->queue.pop_front();
    }
    int err = 0;
    int64_t done = 0;
    char* to = s->direct ? bounce : j.dst;
    if (!to) err = ENOMEM;
    while (!err && done < j.bytes) {
      const ssize_t r = pread(s->fd, to + done, (size_t)(j.bytes - done), (off_t)(j.offset + done));
      if (r < 0 && errno == EINTR) continue;
      if (r <= 0) {
        err = r < 0 ? errno : EIO;  // a short file reads as an I/O error
        break;
      }
      done += r;
    }
    if (!err && s->direct) std::memcpy(j.dst, bounce, (size_t)j.bytes);
    {
      std::lock_guard<std::mutex> lk(s->mu);
      const int slot = (int)(j.ticket % ckv_store::kTickets);
      if (err && !s->failed[slot]) s->failed[slot] = err;
      if (--s->pending[slot] == 0) s->cv_done.notify_all();
    }
  }
}

}  // namespace

int64_t store_keys(const ckv_store* s) { return s->n_keys; }
int64_t store_span_bytes(const ckv_store* s) { return s->span_bytes; }
bool store_direct(const ckv_store* s) { return s->direct; }

ckv_status store_submit(ckv_store* s, const int64_t* keys, int64_t count, char* const* dst,
                        int64_t* ticket) {
  for (int64_t u = 0; u < count; ++u)
    if (keys[u] < 0 || keys[u] >= s->n_keys)
      CKV_FAIL(CKV_EINVAL, "store key %lld outside [0, %lld)", (long long)keys[u], (long long)s->n_keys);
  std::vector<ReadJob> jobs;
  int64_t u = 0;
  while (u < count) {  // a run: consecutive keys into consecutive destinations
    int64_t v = u + 1;
    while (v < count && keys[v] == keys[v - 1] + 1 && dst[v] == dst[v - 1] + s->span_bytes) ++v;
    const int64_t off0 = keys[u] * s->span_bytes, bytes = (v - u) * s->span_bytes;
    for (int64_t p = 0; p < bytes; p += kPieceBytes)
      jobs.push_back(ReadJob{off0 + p, std::min(kPieceBytes, bytes - p), dst[u] + p, 0});
    u = v;
  }
  std::lock_guard<std::mutex> lk(s->mu);
  const int64_t t = s->next_ticket++;
  const int slot = (int)(t % ckv_store::kTickets);
  if (s->pending[slot] != 0) CKV_FAIL(CKV_ESTATE, "too many store reads in flight");
  s->pending[slot] = (int64_t)jobs.size();
  s->failed[slot] = 0;
  for (ReadJob& j : jobs) {
    j.ticket = t;
    s->queue.push_back(j);
  }
  s->cv_work.notify_all();
  *ticket = t;
  return CKV_OK;
}

ckv_status store_wait(ckv_store* s, int64_t ticket) {
  std::unique_lock<std::mutex> lk(s->mu);
  const int slot = (int)(ticket % ckv_store::kTickets);
  s->cv_done.wait(lk, [&] { return s->pending[slot] == 0; });
  const int err = s->failed[slot];
  s->failed[slot] = 0;
  if (err) CKV_FAIL(CKV_EHIP, "store read failed: %s", std::strerror(err));
  return CKV_OK;
}

}  // namespace ckv

using namespace ckv;

extern "C" {

ckv_status ckv_store_open(const char* path, int64_t n_keys, int64_t span_bytes, int32_t io_threads,
                          int32_t flags, ckv_store** out) {
  clear_error();
  if (!out || !path) CKV_FAIL(CKV_EINVAL, "NULL argument");
  *out = nullptr;
  if (n_keys < 1 || span_bytes < 1 || io_threads < 1 || io_threads > 64)
    CKV_FAIL(CKV_EINVAL, "n_keys and span_bytes must be >= 1 and io_threads in [1, 64]");
  if (flags & ~CKV_STORE_DIRECT) CKV_FAIL(CKV_EINVAL, "unknown store flags");
  const bool direct = flags & CKV_STORE_DIRECT;
  if (direct && span_bytes % kDirectAlign)
    CKV_FAIL(CKV_EINVAL, "direct reads need span_bytes a multiple of 4096 (got %lld)", (long long)span_bytes);
  const int fd = open(path, O_RDONLY | (direct ? O_DIRECT : 0));
  if (fd < 0) CKV_FAIL(CKV_EINVAL, "cannot open %s: %s", path, std::strerror(errno));
  const off_t size = lseek(fd, 0, SEEK_END);
  if (size < 0 || (int64_t)size < n_keys * span_bytes) {
    close(fd);
    CKV_FAIL(CKV_EINVAL, "%s holds %lld bytes, fewer than %lld spans of %lld", path, (long long)size,
             (long long)n_keys, (long long)span_bytes);
  }
  ckv_store* s = new (std::nothrow) ckv_store;
  if (!s) {
    close(fd);
    CKV_FAIL(CKV_ENOMEM, "store allocation failed");
  }
  s->fd = fd;
  s->n_keys = n_keys;
  s->span_bytes = span_bytes;
  s->direct = direct;
  try {
    s->pending.assign(ckv_store::kTickets, 0);
    s->failed.assign(ckv_store::kTickets, 0);
    for (int i = 0; i < io_threads; ++i) s->threads.emplace_back(io_worker, s);
  } catch (...) {
    ckv_store_close(s);
    CKV_FAIL(CKV_ENOMEM, "cannot start I/O threads");
  }
  *out = s;
  return CKV_OK;
}

ckv_status ckv_store_close(ckv_store* store) {
  clear_error();
  if (!store) return CKV_OK;
  {
    std::lock_guard<std::mutex> lk(store->mu);
    store->stop = true;
  }
  store->cv_work.notify_all();
  for (std::thread& t : store->threads) t.join();
  if (store->fd >= 0) close(store->fd);
  delete store;
  return CKV_OK;
}

ckv_status ckv_store_read(ckv_store* store, const int64_t* keys, int64_t count, void* dst) {
  clear_error();
  if (!store || count < 0 || (count > 0 && (!keys || !dst))) CKV_FAIL(CKV_EINVAL, "bad argument");
  if (count == 0) return CKV_OK;
  std::vector<char*> d((size_t)count);
  for (int64_t u = 0; u < count; ++u) d[u] = static_cast<char*>(dst) + u * store->span_bytes;
  int64_t t = 0;
  ckv_status s = store_submit(store, keys, count, d.data(), &t);
  if (s != CKV_OK) return s;
  return store_wait(store, t);
}

}  // extern "C"
