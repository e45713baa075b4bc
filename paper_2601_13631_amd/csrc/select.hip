// select.hip -- standalone top-k ContiguousChunk selection (Sec. 4.4).
//
// Up to kSmallKeys scores: one workgroup of 1024 threads holds every key in
// registers (E = 1, 2, 4 or 8 consecutive scores per thread) and runs the
// register-resident radix select of select_regs.h.  Larger m: one 256-thread
// workgroup runs select_topk_block (select_block.h) with the keys cached in
// LDS when m <= kLdsKeys.  Both produce the same set under the same total
// order (score descending, index ascending), ascending.

#include "select_regs.h"

namespace ckv {
namespace {

constexpr int64_t kLdsKeys = 16384;  // 128 KiB of keys
constexpr int kSmallThreads = 1024;
constexpr int64_t kSmallKeys = 8 * kSmallThreads;

template <int THREADS>
__global__ __launch_bounds__(THREADS) void select_kernel(const double* __restrict__ scores,
                                                         int64_t m, int64_t k,
                                                         int32_t* __restrict__ sel, int use_cache) {
  extern __shared__ uint64_t key_cache[];
  __shared__ SelShared sh;
  select_topk_block<THREADS>(scores, m, k, sel, sh, use_cache ? key_cache : nullptr);
}

template <int E>
__global__ __launch_bounds__(kSmallThreads) void select_small_kernel(
    const double* __restrict__ scores, int m, int k, int32_t* __restrict__ sel,
    int32_t* __restrict__ sel_copy) {
  __shared__ RegSelShared<kSmallThreads> sh;
  select_topk_regs<kSmallThreads, E>(scores, m, k, sh, sel, sel_copy);
}

// One workgroup with the keys in registers: select_small_kernel<E>.
template <int E>
void launch_small(const double* scores, int m, int k, int32_t* sel, int32_t* sel_copy,
                  hipStream_t st) {
  hipLaunchKernelGGL(select_small_kernel<E>, dim3(1), dim3(kSmallThreads), 0, st, scores, m, k, sel,
                     sel_copy);
}

}  // namespace

size_t select_ws_bytes(int64_t) { return 0; }

ckv_status launch_select(const double* scores, int64_t m, int64_t k, int32_t* sel, void*, size_t,
                         hipStream_t st, int32_t* sel_copy) {
  if (m <= kSmallKeys) {  // the kernel writes both arrays
    if (m <= kSmallThreads)
      launch_small<1>(scores, (int)m, (int)k, sel, sel_copy, st);
    else if (m <= 2 * kSmallThreads)
      launch_small<2>(scores, (int)m, (int)k, sel, sel_copy, st);
    else if (m <= 4 * kSmallThreads)
      launch_small<4>(scores, (int)m, (int)k, sel, sel_copy, st);
    else
      launch_small<8>(scores, (int)m, (int)k, sel, sel_copy, st);
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
