// select.hip -- standalone top-k ContiguousChunk selection (Sec. 4.4).
//
// Up to kSmallKeys scores: one workgroup holds every key in registers (256
// threads with 4 or 8 consecutive scores each, then 512 and 1024 threads with
// 8) and runs the register-resident radix select of select_regs.h.  Larger m: one 256-thread
// workgroup runs select_topk_block (select_block.h) with the keys cached in
// LDS when m <= kLdsKeys.  Both produce the same set under the same total
// order (score descending, index ascending), ascending.

#include "select_regs.h"

namespace ckv {
namespace {

constexpr int64_t kLdsKeys = 16384;  // 128 KiB of keys
constexpr int64_t kSmallKeys = 8 * 1024;  // 1024 threads, 8 keys each

template <int THREADS>
__global__ __launch_bounds__(THREADS) void select_kernel(const double* __restrict__ scores,
                                                         int64_t m, int64_t k,
                                                         int32_t* __restrict__ sel, int use_cache) {
  extern __shared__ uint64_t key_cache[];
  __shared__ SelShared sh;
  select_topk_block<THREADS>(scores, m, k, sel, sh, use_cache ? key_cache : nullptr);
}

template <int THREADS, int E>
__global__ __launch_bounds__(THREADS) void select_small_kernel(
    const double* __restrict__ scores, int m, int k, int32_t* __restrict__ sel,
    int32_t* __restrict__ sel_copy) {
  __shared__ RegSelShared<THREADS> sh;
  select_topk_regs<THREADS, E>(scores, m, k, sh, sel, sel_copy);
}

// One workgroup of THREADS threads with E keys each in registers.
template <int THREADS, int E>
void launch_small(const double* scores, int m, int k, int32_t* sel, int32_t* sel_copy,
                  hipStream_t st) {
  hipLaunchKernelGGL((select_small_kernel<THREADS, E>), dim3(1), dim3(THREADS), 0, st, scores, m,
                     k, sel, sel_copy);
}

}  // namespace

size_t select_ws_bytes(int64_t) { return 0; }

ckv_status launch_select(const double* scores, int64_t m, int64_t k, int32_t* sel, void*, size_t,
                         hipStream_t st, int32_t* sel_copy) {
  if (m <= kSmallKeys) {  // the kernel writes both arrays
    // the fewest waves that hold the keys at up to 8 per thread: per round
    // every wave counts its digits and meets the others at two barriers, so
    // fewer, fuller waves finish a round sooner
    if (m <= 1024) launch_small<256, 4>(scores, (int)m, (int)k, sel, sel_copy, st);
    else if (m <= 2048) launch_small<256, 8>(scores, (int)m, (int)k, sel, sel_copy, st);
    else if (m <= 4096) launch_small<512, 8>(scores, (int)m, (int)k, sel, sel_copy, st);
    else launch_small<1024, 8>(scores, (int)m, (int)k, sel, sel_copy, st);
    CKV_HIP(hipGetLastError());
    return CKV_OK;
  }
  const int use_cache = m <= kLdsKeys;
  const size_t shmem = use_cache ? (size_t)m * sizeof(uint64_t) : 0;
  // raise the dynamic LDS limit once (thread-safe static initialisation)
  static const hipError_t attr = hipFuncSetAttribute(
      (const void*)select_kernel<256>, hipFuncAttributeMaxDynamicSharedMemorySize,
      (int)(kLdsKeys * sizeof(uint64_t)));
  CKV_HIP(attr);
  hipLaunchKernelGGL(select_kernel<256>, dim3(1), dim3(256), shmem, st, scores, m, k, sel,
                     use_cache);
  CKV_HIP(hipGetLastError());
  if (sel_copy)
    CKV_HIP(hipMemcpyAsync(sel_copy, sel, (size_t)k * sizeof(int32_t), hipMemcpyDeviceToDevice, st));
  return CKV_OK;
}

}  // namespace ckv
