// select_regs.h -- top-k ContiguousChunk selection (Sec. 4.4) by one
// workgroup of THREADS threads holding every key in registers (E consecutive
// scores per thread).
//
// Keeps the k largest of m fp64 chunk scores under the total order (score
// descending, index ascending) and writes their indices in ascending order.
// A radix select on order-preserving 64-bit keys (select_block.h's order_key)
// with 4-bit digits whose counts come from packed per-lane counters summed by
// DPP and the permlane swaps (no ballots: 16 masks per key in scalar registers
// queue every wave on the CU's scalar unit; no LDS atomics: the chunk scores
// of a layer share their high bits, so per-bin atomics would all collide):
// the first digit ends at the highest bit where the smallest and
// largest key differ, every later one is the next 4 bits down; the search ends
// when the chosen digit holds exactly the keys still needed or the last bit
// is fixed (then the lowest indices win).  The ordered compaction counts with
// ballots.  Reductions use DPP and the gfx950 permlane swaps.

#pragma once

#include "select_block.h"

namespace ckv {

template <int THREADS>
struct RegSelShared {
  static constexpr int kWaves = THREADS / 64;
  uint32_t whist[kWaves][16];  // per-wave digit counts of the round
  uint64_t wlo[kWaves], whi[kWaves];
  uint32_t wgt[kWaves], weq[kWaves];
  uint64_t prefix, mask;
  int32_t remaining, done;
};

__device__ __forceinline__ void minmax_with(uint64_t& lo, uint64_t& hi, uint64_t plo, uint64_t phi) {
  lo = plo < lo ? plo : lo;
  hi = phi > hi ? phi : hi;
}

// Wave minimum of lo and maximum of hi, in every lane.
__device__ __forceinline__ void wave_minmax(uint64_t& lo, uint64_t& hi) {
  minmax_with(lo, hi, dpp64<kDppQuadXor1>(lo), dpp64<kDppQuadXor1>(hi));
  minmax_with(lo, hi, dpp64<kDppQuadXor2>(lo), dpp64<kDppQuadXor2>(hi));
  minmax_with(lo, hi, dpp64<kDppRowHalfMirror>(lo), dpp64<kDppRowHalfMirror>(hi));
  minmax_with(lo, hi, dpp64<kDppRowMirror>(lo), dpp64<kDppRowMirror>(hi));
  uint64_t la, lb, ha, hb;
  swap_pair64<16>(lo, la, lb);
  swap_pair64<16>(hi, ha, hb);
  lo = la;
  hi = ha;
  minmax_with(lo, hi, lb, hb);
  swap_pair64<32>(lo, la, lb);
  swap_pair64<32>(hi, ha, hb);
  lo = la;
  hi = ha;
  minmax_with(lo, hi, lb, hb);
}

// x + (x of lane l ^ 16) and x + (x of lane l ^ 32): the swaps hand each lane
// its own value and its partner's, in some order, and the sum is symmetric.
__device__ __forceinline__ uint32_t pair_sum16(uint32_t x) {
  const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  return r[0] + r[1];
}
__device__ __forceinline__ uint32_t pair_sum32(uint32_t x) {
  const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return r[0] + r[1];
}

// The wave's count of keys per digit value 0..15 (digit 16: not a candidate),
// for E keys per lane: each lane counts its digits in
// 4-bit fields of one 64-bit word (E <= 15), the fields are spread to bytes
// and summed over each row of 16 lanes by DPP (at most 16 * E <= 255), then
// widened to 16-bit fields and summed over the four rows by the permlane
// swaps.  Lane 15 returns digit pair (2i, 2i + 1) in cnt[i] (low, high half).
template <int E>
__device__ __forceinline__ void wave_digit_counts(const int (&cd)[E], uint32_t (&cnt)[8]) {
  static_assert(E <= 15, "4-bit per-lane fields");
  uint64_t acc = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) acc += cd[e] < 16 ? 1ull << (4 * cd[e]) : 0ull;
  const uint32_t lo = (uint32_t)acc, hi = (uint32_t)(acc >> 32);
  // byte j of by[q]: digit 8 * (q / 2) + 2 * j + (q % 2)
  uint32_t by[4] = {lo & 0x0F0F0F0Fu, (lo >> 4) & 0x0F0F0F0Fu, hi & 0x0F0F0F0Fu,
                    (hi >> 4) & 0x0F0F0F0Fu};
#pragma unroll
  for (int q = 0; q < 4; ++q) {  // inclusive sums along the row: lane 15 holds the row's
    by[q] += dpp32<kDppRowShr1>(by[q]);
    by[q] += dpp32<kDppRowShr2>(by[q]);
    by[q] += dpp32<kDppRowShr4>(by[q]);
    by[q] += dpp32<kDppRowShr8>(by[q]);
  }
  // 16-bit fields: cnt[i] = (digit 2i, digit 2i + 1); by[q] byte j is digit
  // 8 * (q / 2) + 2 * j + (q % 2), so digit pair i = 4 * (q / 2) + j comes from
  // byte j of by[2 * (q / 2)] (even digit) and of by[2 * (q / 2) + 1] (odd)
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t ev = (by[2 * h] >> (8 * j)) & 0xFFu, od = (by[2 * h + 1] >> (8 * j)) & 0xFFu;
      cnt[4 * h + j] = pair_sum32(pair_sum16(ev | (od << 16)));
    }
}

// Called by all THREADS threads; m <= E * THREADS, 1 <= k <= m, 4 <= E <= 15.  Thread t
// holds scores t*E .. t*E+E-1.  The k indices go to out0[0..k) and, when
// out1 is not null, to out1 too (each thread writes its own kept indices).
template <int THREADS, int E>
__device__ __forceinline__ void select_topk_regs(const double* __restrict__ scores, int m, int k,
                                                 RegSelShared<THREADS>& sh, int32_t* out0,
                                                 int32_t* out1) {
  static_assert(E >= 4 && E <= 15, "keys per thread");
  constexpr int kWaves = THREADS / 64;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i0 = tid * E;
  uint64_t x[E];
  bool valid[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    valid[e] = i0 + e < m;
    x[e] = order_key(scores[min(i0 + e, m - 1)]);  // unconditional load
  }
  uint64_t lo = ~0ull, hi = 0;
#pragma unroll
  for (int e = 0; e < E; ++e)
    if (valid[e]) {
      lo = x[e] < lo ? x[e] : lo;
      hi = x[e] > hi ? x[e] : hi;
    }
  wave_minmax(lo, hi);
  if (lane == 0) {
    sh.wlo[wave] = lo;
    sh.whi[wave] = hi;
  }
  __syncthreads();
#pragma unroll
  for (int w = 0; w < kWaves; ++w) minmax_with(lo, hi, sh.wlo[w], sh.whi[w]);

  uint64_t prefix, mask;
  int remaining = k;
  if (lo == hi) {  // every key equal: the lowest indices win
    prefix = lo;
    mask = ~0ull;
  } else {
    const int top = 63 - __clzll(lo ^ hi);
    int shift = top >= 3 ? top - 3 : 0;
    mask = shift + 4 >= 64 ? 0 : ~((1ull << (shift + 4)) - 1);  // bits above the window: shared
    prefix = lo & mask;
    for (;;) {
      // this wave's count of candidates per digit value, digit b in lane b
      // (cd = 16: not a candidate)
      int cd[E];
#pragma unroll
      for (int e = 0; e < E; ++e)
        cd[e] = valid[e] && (x[e] & mask) == prefix ? (int)((x[e] >> shift) & 15) : 16;
      {
        uint32_t cnt[8];
        wave_digit_counts<E>(cd, cnt);
        if (lane == 15)
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            sh.whist[wave][2 * i] = cnt[i] & 0xFFFFu;
            sh.whist[wave][2 * i + 1] = cnt[i] >> 16;
          }
      }
      __syncthreads();
      if (wave == 0) {
        // lane i < 16 takes digit 15 - i; inclusive scan over i gives the
        // count of candidates in digits >= 15 - i
        uint32_t tot = 0;
        if (lane < 16)
#pragma unroll
          for (int w = 0; w < kWaves; ++w) tot += sh.whist[w][lane];
        const uint32_t u = dpp32<kDppRowMirror>(tot);
        uint32_t cum = u;
        cum += dpp32<kDppRowShr1>(cum);
        cum += dpp32<kDppRowShr2>(cum);
        cum += dpp32<kDppRowShr4>(cum);
        cum += dpp32<kDppRowShr8>(cum);
        const uint32_t before = cum - u;
        if (lane < 16 && before < (uint32_t)remaining && cum >= (uint32_t)remaining) {
          const uint64_t digit = (uint64_t)(15 - lane);
          sh.prefix = prefix | (digit << shift);
          sh.mask = mask | (15ull << shift);
          sh.remaining = remaining - (int)before;
          sh.done = u == (uint32_t)(remaining - (int)before) || shift == 0;
        }
      }
      __syncthreads();
      prefix = sh.prefix;
      mask = sh.mask;
      remaining = sh.remaining;
      if (sh.done) break;
      shift = shift >= 4 ? shift - 4 : 0;
    }
  }

  // ascending compaction: key i is kept if (key & mask) > prefix, or equal and
  // among the first `remaining` equal keys by index.  Counts of greater and of
  // equal keys before this thread's first key: wave ballots, then the waves
  // before it (one barrier).
  bool gt[E], eq[E];
  const uint64_t below = (1ull << lane) - 1;
  uint32_t gt_wave = 0, eq_wave = 0, gt_lane = 0, eq_lane = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const uint64_t xm = x[e] & mask;
    gt[e] = valid[e] && xm > prefix;
    eq[e] = valid[e] && xm == prefix;
    const uint64_t bg = __ballot(gt[e]), be = __ballot(eq[e]);
    gt_wave += __popcll(bg);
    eq_wave += __popcll(be);
    gt_lane += __popcll(bg & below);
    eq_lane += __popcll(be & below);
  }
  if (lane == 0) {
    sh.wgt[wave] = gt_wave;
    sh.weq[wave] = eq_wave;
  }
  __syncthreads();
  uint32_t gt_before = gt_lane, eq_before = eq_lane;
  for (int w = 0; w < wave; ++w) {
    gt_before += sh.wgt[w];
    eq_before += sh.weq[w];
  }
  int eq_rank = (int)eq_before;
  int pos = (int)gt_before + min((int)eq_before, remaining);
#pragma unroll
  for (int e = 0; e < E; ++e) {
    bool take = gt[e];
    if (eq[e]) take = eq_rank++ < remaining;
    if (take) {
      out0[pos] = i0 + e;
      if (out1) out1[pos] = i0 + e;
      ++pos;
    }
  }
}

}  // namespace ckv
