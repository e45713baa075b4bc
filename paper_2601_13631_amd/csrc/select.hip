// select.hip -- top-k ContiguousChunk selection (Sec. 4.4) for gfx950.
//
// Keeps the k largest of m fp64 chunk scores under the total order (score
// descending, index ascending) and writes their indices in ascending order.
//
// One workgroup of 1024 threads runs a radix select on 64-bit order-preserving
// keys (sign-flipped IEEE bits, -0.0 folded onto +0.0, NaN below -inf).  Each
// round first reduces the smallest and largest key still in play; the highest
// bit where they differ starts the round's 8-bit digit, so rounds never waste
// a histogram on bits every candidate shares.  The digit histogram lives in
// LDS (integer atomics: exact, order-independent).  A round ends the search
// when the chosen bin holds exactly the number of keys still needed, or when
// all candidates are equal; the lowest indices then win among equal keys.
// Output is an in-order compaction with block-wide exclusive scans, so the
// indices come out ascending and the result depends only on the score bits.
//
// For m <= kLdsKeys the keys are cached in LDS; larger m re-reads the scores.

#include "ckv_internal.h"

namespace ckv {
namespace {

constexpr int kThreads = 1024;
constexpr int kWavesSel = kThreads / 64;
constexpr int64_t kLdsKeys = 16384;  // 128 KiB of keys

__device__ __forceinline__ uint64_t order_key(double x) {
  uint64_t u = (uint64_t)__double_as_longlong(x);
  if ((u << 1) == 0) u = 0;                        // -0.0 -> +0.0
  if ((u & 0x7FF0000000000000ull) == 0x7FF0000000000000ull && (u & 0x000FFFFFFFFFFFFFull))
    return 0;                                      // NaN: below everything
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// block-wide minimum of lo and maximum of hi (every thread gets both)
__device__ void block_minmax(uint64_t& lo, uint64_t& hi, uint64_t* red_lo, uint64_t* red_hi) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint64_t l2 = __shfl_xor(lo, off), h2 = __shfl_xor(hi, off);
    lo = l2 < lo ? l2 : lo;
    hi = h2 > hi ? h2 : hi;
  }
  __syncthreads();
  if (lane == 0) { red_lo[wave] = lo; red_hi[wave] = hi; }
  __syncthreads();
  lo = red_lo[0];
  hi = red_hi[0];
  for (int w = 1; w < kWavesSel; ++w) {
    lo = red_lo[w] < lo ? red_lo[w] : lo;
    hi = red_hi[w] > hi ? red_hi[w] : hi;
  }
}

// exclusive prefix sum over the block (returns this thread's exclusive prefix)
__device__ int64_t block_exclusive_scan(int64_t v, int64_t* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int64_t x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    int64_t y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  __syncthreads();
  if (lane == 63) red[wave] = x;
  __syncthreads();
  int64_t before = 0;
  for (int w = 0; w < wave; ++w) before += red[w];
  return before + x - v;
}

struct SelState {
  uint64_t prefix, mask;
  int64_t remaining;
  int done;
};

__global__ __launch_bounds__(kThreads) void select_kernel(const double* __restrict__ scores,
                                                          int64_t m, int64_t k,
                                                          int32_t* __restrict__ sel,
                                                          int use_lds) {
  extern __shared__ uint64_t key_cache[];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t wsum[4];
  __shared__ uint64_t red_u[kWavesSel];
  __shared__ uint64_t red_u2[kWavesSel];
  __shared__ int64_t red_i[kWavesSel];
  __shared__ SelState st;

  const int tid = threadIdx.x;
  if (use_lds)
    for (int64_t i = tid; i < m; i += kThreads) key_cache[i] = order_key(scores[i]);
  if (tid == 0) {
    st.prefix = 0;
    st.mask = 0;
    st.remaining = k;
    st.done = 0;
  }
  __syncthreads();
  auto key_at = [&](int64_t i) -> uint64_t {
    return use_lds ? key_cache[i] : order_key(scores[i]);
  };

  for (int round = 0; round < 64; ++round) {
    const uint64_t prefix = st.prefix, mask = st.mask;
    // smallest and largest key among the candidates
    uint64_t lo = ~0ull, hi = 0;
    for (int64_t i = tid; i < m; i += kThreads) {
      uint64_t x = key_at(i);
      if ((x & mask) == prefix) { lo = x < lo ? x : lo; hi = x > hi ? x : hi; }
    }
    block_minmax(lo, hi, red_u, red_u2);
    if (lo == hi) {  // every candidate equal: the lowest indices among them win
      if (tid == 0) { st.prefix = lo; st.mask = ~0ull; st.done = 1; }
      __syncthreads();
      break;
    }
    const int top = 63 - __clzll(lo ^ hi);
    const int shift = top >= 7 ? top - 7 : 0;
    for (int b = tid; b < 256; b += kThreads) hist[b] = 0;
    __syncthreads();
    for (int64_t i = tid; i < m; i += kThreads) {
      uint64_t x = key_at(i);
      if ((x & mask) == prefix) atomicAdd(&hist[(x >> shift) & 255], 1u);
    }
    __syncthreads();
    // counts of keys in bins >= b, as an inclusive scan over t = 255 - b by the
    // first four waves; the bin where that count first reaches `need` is chosen
    const int64_t need = st.remaining;
    uint32_t cum = 0, mine = 0;
    if (tid < 256) {
      mine = hist[255 - tid];
      cum = mine;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t y = __shfl_up(cum, off);
        if ((tid & 63) >= off) cum += y;
      }
      if ((tid & 63) == 63) wsum[tid >> 6] = cum;
    }
    __syncthreads();
    if (tid < 256) {
      for (int w = 0; w < (tid >> 6); ++w) cum += wsum[w];
      const uint32_t before = cum - mine;
      if (before < need && cum >= need) {  // exactly one thread
        const int b = 255 - tid;
        const uint64_t digit_mask = 255ull << shift;
        const uint64_t keep_hi = shift + 8 >= 64 ? 0 : ~((1ull << (shift + 8)) - 1);
        st.prefix = (lo & keep_hi) | ((uint64_t)b << shift);
        st.mask = keep_hi | digit_mask;
        st.remaining = need - before;
        st.done = (mine == (uint32_t)st.remaining) || shift == 0;
      }
    }
    __syncthreads();
    if (st.done) break;
  }

  // ascending compaction: i is kept if (key & mask) > prefix, or equal and among
  // the first `remaining` equal keys by index
  const uint64_t prefix = st.prefix, mask = st.mask;
  const int64_t remaining = st.remaining;
  const int64_t per = (m + kThreads - 1) / kThreads;
  const int64_t i0 = (int64_t)tid * per, i1 = min(m, i0 + per);
  int64_t n_gt = 0, n_eq = 0;
  for (int64_t i = i0; i < i1; ++i) {
    uint64_t x = key_at(i) & mask;
    n_gt += x > prefix;
    n_eq += x == prefix;
  }
  const int64_t gt_before = block_exclusive_scan(n_gt, red_i);
  const int64_t eq_before = block_exclusive_scan(n_eq, red_i);
  int64_t eq_rank = eq_before;
  int64_t pos = gt_before + min(eq_before, remaining);
  for (int64_t i = i0; i < i1; ++i) {
    uint64_t x = key_at(i) & mask;
    bool take = x > prefix;
    if (x == prefix) take = eq_rank++ < remaining;
    if (take) sel[pos++] = (int32_t)i;
  }
}

}  // namespace

size_t select_ws_bytes(int64_t) { return 0; }

ckv_status launch_select(const double* scores, int64_t m, int64_t k, int32_t* sel, void*, size_t,
                         hipStream_t st) {
  const int use_lds = m <= kLdsKeys;
  const size_t shmem = use_lds ? (size_t)m * sizeof(uint64_t) : 0;
  // raise the dynamic LDS limit once (thread-safe static initialisation)
  static const hipError_t attr = hipFuncSetAttribute(
      (const void*)select_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
      (int)(kLdsKeys * sizeof(uint64_t)));
  CKV_HIP(attr);
  hipLaunchKernelGGL(select_kernel, dim3(1), dim3(kThreads), shmem, st, scores, m, k, sel, use_lds);
  CKV_HIP(hipGetLastError());
  return CKV_OK;
}

}  // namespace ckv
