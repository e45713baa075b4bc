// select_block.h -- top-k ContiguousChunk selection (Sec. 4.4) by one
// workgroup of THREADS threads (a multiple of 64; one wave suits small m, where
// the workgroup barriers then cost almost nothing).
//
// Keeps the k largest of m fp64 chunk scores under the total order (score
// descending, index ascending) and writes their indices in ascending order.
// Radix select on 64-bit order-preserving keys (sign-flipped IEEE bits, -0.0
// folded onto +0.0, NaN below -inf).  Each round histograms an 8-bit digit that
// starts at the highest bit where the smallest and largest candidate differ, so
// no round is spent on bits every candidate shares; after the bin is chosen, a
// block-wide min/max over its keys bounds the next round's candidates.  The
// search ends when the chosen bin holds exactly the keys still needed or all
// candidates are equal; the lowest indices then win among equal keys.  Output
// is an in-order compaction with one block-wide exclusive scan (the counts of
// greater and of equal keys packed in one 64-bit word), so the indices come
// out ascending.  Every count is an integer (LDS atomics): the result depends
// only on the score bits.  With a key cache (LDS, m entries) the scores are
// read from global memory once; without one, every pass re-reads them (they
// stay in L2).

#pragma once

#include "ckv_internal.h"

namespace ckv {

constexpr int kSelMaxWaves = 4;

__device__ __forceinline__ uint64_t order_key(double x) {
  uint64_t u = (uint64_t)__double_as_longlong(x);
  if ((u << 1) == 0) u = 0;  // -0.0 -> +0.0
  if ((u & 0x7FF0000000000000ull) == 0x7FF0000000000000ull && (u & 0x000FFFFFFFFFFFFFull))
    return 0;  // NaN: below everything
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

struct SelShared {
  uint32_t hist[256];
  uint32_t wsum[4];
  uint64_t red_lo[kSelMaxWaves], red_hi[kSelMaxWaves];
  int64_t red_i[kSelMaxWaves];
  uint64_t prefix, mask, lo, hi;
  int64_t remaining;
  int done;
};

// Block-wide minimum of lo and maximum of hi, left in sh.lo / sh.hi.
template <int THREADS>
__device__ __forceinline__ void sel_block_minmax(uint64_t lo, uint64_t hi, SelShared& sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint64_t l2 = __shfl_xor(lo, off), h2 = __shfl_xor(hi, off);
    lo = l2 < lo ? l2 : lo;
    hi = h2 > hi ? h2 : hi;
  }
  if (lane == 0) { sh.red_lo[wave] = lo; sh.red_hi[wave] = hi; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < THREADS / 64; ++w) {
      lo = sh.red_lo[w] < lo ? sh.red_lo[w] : lo;
      hi = sh.red_hi[w] > hi ? sh.red_hi[w] : hi;
    }
    sh.lo = lo;
    sh.hi = hi;
  }
  __syncthreads();
}

// Exclusive prefix sum over the block (this thread's exclusive prefix).
template <int THREADS>
__device__ __forceinline__ int64_t sel_block_exclusive_scan(int64_t v, SelShared& sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int64_t x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int64_t y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  __syncthreads();  // red_i may still be read by a previous scan
  if (lane == 63) sh.red_i[wave] = x;
  __syncthreads();
  int64_t before = 0;
  for (int w = 0; w < wave; ++w) before += sh.red_i[w];
  return before + x - v;
}

// Called by all THREADS threads of the workgroup; 1 <= k <= m.  cache:
// nullptr, or LDS room for m keys.
template <int THREADS>
__device__ __forceinline__ void select_topk_block(const double* scores, int64_t m, int64_t k,
                                                  int32_t* sel, SelShared& sh, uint64_t* cache) {
  static_assert(THREADS % 64 == 0 && THREADS <= 64 * kSelMaxWaves, "1 to 4 waves");
  const int tid = threadIdx.x;
  auto key_at = [&](int64_t i) -> uint64_t { return cache ? cache[i] : order_key(scores[i]); };
  {
    uint64_t lo = ~0ull, hi = 0;
    for (int64_t i = tid; i < m; i += THREADS) {
      const uint64_t x = order_key(scores[i]);
      if (cache) cache[i] = x;
      lo = x < lo ? x : lo;
      hi = x > hi ? x : hi;
    }
    sel_block_minmax<THREADS>(lo, hi, sh);  // its barriers also publish the cache
  }
  if (tid == 0) {
    sh.prefix = 0;
    sh.mask = 0;
    sh.remaining = k;
    sh.done = 0;
  }
  __syncthreads();
  for (int round = 0; round < 64; ++round) {
    const uint64_t lo = sh.lo, hi = sh.hi, prefix = sh.prefix, mask = sh.mask;
    if (lo == hi) {  // every candidate equal: the lowest indices among them win
      __syncthreads();
      if (tid == 0) { sh.prefix = lo; sh.mask = ~0ull; }
      __syncthreads();
      break;
    }
    const int top = 63 - __clzll(lo ^ hi);
    const int shift = top >= 7 ? top - 7 : 0;
    for (int b = tid; b < 256; b += THREADS) sh.hist[b] = 0;
    __syncthreads();
    for (int64_t i = tid; i < m; i += THREADS) {
      const uint64_t x = key_at(i);
      if ((x & mask) == prefix) atomicAdd(&sh.hist[(int)((x >> shift) & 255)], 1u);
    }
    __syncthreads();
    // count of candidates in bins >= b as an inclusive scan over t = 255 - b
    // (thread i holds t = i*kPer .. i*kPer+kPer-1); the bin where that count
    // first reaches `need` is chosen (one thread)
    constexpr int kPer = 256 / THREADS;
    const int64_t need = sh.remaining;
    uint32_t cnt[kPer];
    uint32_t own = 0;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      cnt[q] = sh.hist[255 - (tid * kPer + q)];
      own += cnt[q];
    }
    uint32_t cum = own;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const uint32_t y = __shfl_up(cum, off);
      if ((tid & 63) >= off) cum += y;
    }
    if (THREADS > 64) {
      if ((tid & 63) == 63) sh.wsum[tid >> 6] = cum;
      __syncthreads();
      for (int w = 0; w < (tid >> 6); ++w) cum += sh.wsum[w];
    }
    uint32_t before = cum - own;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const uint32_t after = before + cnt[q];
      if (before < need && after >= need) {
        const int b = 255 - (tid * kPer + q);
        const uint64_t keep_hi = shift + 8 >= 64 ? 0 : ~((1ull << (shift + 8)) - 1);
        sh.prefix = (lo & keep_hi) | ((uint64_t)b << shift);
        sh.mask = keep_hi | (255ull << shift);
        sh.remaining = need - before;
        sh.done = (cnt[q] == (uint32_t)sh.remaining) || shift == 0;
      }
      before = after;
    }
    __syncthreads();
    if (sh.done) break;
    // bounds of the chosen bin's keys for the next round
    {
      const uint64_t p2 = sh.prefix, m2 = sh.mask;
      uint64_t blo = ~0ull, bhi = 0;
      for (int64_t i = tid; i < m; i += THREADS) {
        const uint64_t x = key_at(i);
        if ((x & m2) == p2) {
          blo = x < blo ? x : blo;
          bhi = x > bhi ? x : bhi;
        }
      }
      sel_block_minmax<THREADS>(blo, bhi, sh);
    }
  }

  // ascending compaction: i is kept if (key & mask) > prefix, or equal and among
  // the first `remaining` equal keys by index
  const uint64_t prefix = sh.prefix, mask = sh.mask;
  const int64_t remaining = sh.remaining;
  const int64_t per = (m + THREADS - 1) / THREADS;
  const int64_t i0 = min(m, (int64_t)tid * per), i1 = min(m, i0 + per);
  int64_t n_gt = 0, n_eq = 0;
  for (int64_t i = i0; i < i1; ++i) {
    const uint64_t x = key_at(i) & mask;
    n_gt += x > prefix;
    n_eq += x == prefix;
  }
  // one scan of both counts: greater in the high 32 bits, equal in the low
  // (m < 2^31, so neither field carries into the other)
  const int64_t both = sel_block_exclusive_scan<THREADS>((n_gt << 32) | n_eq, sh);
  const int64_t gt_before = both >> 32, eq_before = both & 0xffffffffll;
  int64_t eq_rank = eq_before;
  int64_t pos = gt_before + min(eq_before, remaining);
  for (int64_t i = i0; i < i1; ++i) {
    const uint64_t x = key_at(i) & mask;
    bool take = x > prefix;
    if (x == prefix) take = eq_rank++ < remaining;
    if (take) sel[pos++] = (int32_t)i;
  }
}

}  // namespace ckv
