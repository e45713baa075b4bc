// select.hip -- standalone top-k ContiguousChunk selection (Sec. 4.4): one
// workgroup runs the block selection of select_block.h over the m scores,
// with the keys cached in LDS when m <= kLdsKeys.  (Four waves: a single wave
// measured slower even for m = 1024.)

#include "select_block.h"

namespace ckv {
namespace {

constexpr int64_t kLdsKeys = 16384;  // 128 KiB of keys

template <int THREADS>
__global__ __launch_bounds__(THREADS) void select_kernel(const double* __restrict__ scores,
                                                         int64_t m, int64_t k,
                                                         int32_t* __restrict__ sel, int use_cache) {
  extern __shared__ uint64_t key_cache[];
  __shared__ SelShared sh;
  select_topk_block<THREADS>(scores, m, k, sel, sh, use_cache ? key_cache : nullptr);
}

}  // namespace

size_t select_ws_bytes(int64_t) { return 0; }

ckv_status launch_select(const double* scores, int64_t m, int64_t k, int32_t* sel, void*, size_t,
                         hipStream_t st) {
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
  return CKV_OK;
}

}  // namespace ckv
