// score.hip -- chunk scoring (Sec. 4.4, Eq. 1) for gfx950.
//
// A_j = sum over rows r=(t,h) of sum_{i in chunk j} p_{r,i},
// p_{r,i} = softmax_i(sm_scale * q_r . k_i) over the n prefix keys.
//
// Work split.  Rows of one KV head g are r = t*G + i (query t, head g*G+i).  A
// workgroup owns 256 rows (4 waves x 64) of one KV head and one key range of
// `key_range` keys.  Each wave keeps its 64 query rows in registers as the B
// operand of bf16 MFMA 32x32x16 and streams the range's keys through LDS in
// 32-key subtiles, computing S^T = K Q^T so that every lane owns one query row
// and holds 16 of the 32 keys of a subtile (its partner lane l^32 the other 16).
//
// Softmax without a second pass.  Each row takes as reference mc the scaled
// maximum of its logits over the prefix's first 32 keys (every workgroup of
// the row computes the same value) and each (row, range) accumulates, per
// chunk, P = sum exp2(c1*dot - mc) (c1 = sm_scale*log2 e) in fp32 over at most
// one chunk, plus z = sum of the range's chunk sums in fp64.  Finalize kernels
// fold the ranges of a row in fp64: Z = sum z, w = 1/Z, A_j = sum_r w P.  The
// result is exact in real arithmetic for any reference; the reference only has
// to keep exp2 finite.  If any chunk sum of a range is not finite the
// workgroup recomputes that range against its own exact maximum (two passes),
// and the fold rescales that range by exp2(mc - max mc), so the fast path never
// trades correctness for speed.
//
// All sums have a fixed order: results are bitwise reproducible run to run.

#include <cfloat>

#include "ckv_internal.h"

namespace ckv {
namespace {

constexpr int kWaves = 4;
constexpr int kWaveRows = 64;
constexpr int kBlockRows = kWaves * kWaveRows;  // 256
constexpr int kSub = 32;                        // keys per subtile
constexpr float kOverflowGuard = 0x1p100f;      // a chunk sum above this forces the exact pass
constexpr int kFallbackBlocks = 64;             // grid of the (almost always idle) fallback kernel

enum ChunkMode { kC4 = 0, kC8 = 1, kC16 = 2, kC32 = 3, kC32x = 4 };  // kC32x: c = 64, 96, ...

__device__ __forceinline__ float partner_f(float x) {
  // value of the same register in lane l^32
  int v = __float_as_int(x);
  auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return __int_as_float(threadIdx.x & 32 ? r[0] : r[1]);
}

__device__ __forceinline__ double partner_d(double x) {
  int2 v = *reinterpret_cast<int2*>(&x);
  auto rx = __builtin_amdgcn_permlane32_swap(v.x, v.x, false, false);
  auto ry = __builtin_amdgcn_permlane32_swap(v.y, v.y, false, false);
  int2 o;
  o.x = threadIdx.x & 32 ? rx[0] : rx[1];
  o.y = threadIdx.x & 32 ? ry[0] : ry[1];
  return *reinterpret_cast<double*>(&o);
}

// ---------------------------------------------------------------------------
// bf16 main kernel
// ---------------------------------------------------------------------------
// LDS subtile: 32 keys x D bf16, 16-byte segments XOR-swizzled by key so that
// the MFMA operand reads (consecutive lanes = consecutive keys, same segment)
// hit distinct banks for both 8- and 16-lane bank cycles.
template <int D>
struct SubtileLds {
  static constexpr int kSegs = D / 8;  // 16-byte segments per key row
  __device__ static int offset(int key, int seg) {  // in bf16 elements
    return key * D + ((seg ^ ((key ^ (key >> 3)) & (kSegs - 1))) * 8);
  }
};

struct ScoreArgs {
  const uint16_t* q;   // [S][Hq][D] bf16 bits
  const uint16_t* k;   // [n][Hkv][D]
  float* part;         // [Hkv][NR][CPR][ldp]: rows padded to whole row blocks
  float* mc;           // [Hkv][NR][R]
  double* z;           // [Hkv][NR][R]
  int* flags;          // [nblocks]: the range overflowed in the main pass
  int64_t n;
  int S, Hq, Hkv, G, R, ldp, c, key_range, n_ranges, cpr, n_row_blocks;
  float c1;            // sm_scale * log2(e)
  uint32_t nblocks, nblocks_padded;
};

constexpr int kStage = 64;  // keys per LDS stage: two 32-key subtiles

// The next stage's K rows are fetched into registers while the current stage is
// consumed from LDS, then written to the other LDS buffer: one barrier per stage.
// Loads are unconditional (rows past the range end read the stage's first row
// and are zeroed when stored), so the compiler never has to wait on them early.
template <int D>
struct StageRegs {
  static constexpr int kPer = kStage * (D / 8) / (kWaves * 64);  // 16-byte loads per thread
  u32x4 v[kPer];
  uint32_t valid;  // bit p: piece p is inside the range
};

template <int D>
__device__ __forceinline__ void stage_load(const uint16_t* kstage, int64_t keys_left,
                                           const uint32_t (&voff)[StageRegs<D>::kPer],
                                           const uint32_t (&voff0)[StageRegs<D>::kPer],
                                           StageRegs<D>& r) {
  constexpr int kSegs = D / 8;
  r.valid = 0;
#pragma unroll
  for (int p = 0; p < StageRegs<D>::kPer; ++p) {
    const int key = (threadIdx.x + p * kWaves * 64) / kSegs;
    const bool ok = key < keys_left;
    r.valid |= (ok ? 1u : 0u) << p;
    r.v[p] = *reinterpret_cast<const u32x4*>(kstage + (ok ? voff[p] : voff0[p]));
  }
}

template <int D>
__device__ __forceinline__ void stage_store(const StageRegs<D>& r, uint16_t* lds) {
  constexpr int kSegs = D / 8;
#pragma unroll
  for (int p = 0; p < StageRegs<D>::kPer; ++p) {
    const int idx = threadIdx.x + p * kWaves * 64;
    u32x4 v = r.v[p];
    if (!((r.valid >> p) & 1u)) v = u32x4{0u, 0u, 0u, 0u};
    *reinterpret_cast<u32x4*>(lds + SubtileLds<D>::offset(idx / kSegs, idx % kSegs)) = v;
  }
}

// Per-chunk sums of one subtile for one row tile, combined across the lane pair.
// Fills sums[] (how many depends on the mode) in the order of chunk index.
template <int MODE>
__device__ __forceinline__ void chunk_sums(const f32x16& p, float* sums) {
  if constexpr (MODE == kC32 || MODE == kC32x) {
    float s = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) s += p[v];
    sums[0] = s + partner_f(s);
  } else if constexpr (MODE == kC16) {
    float s0 = 0.f, s1 = 0.f;
#pragma unroll
    for (int v = 0; v < 8; ++v) { s0 += p[v]; s1 += p[v + 8]; }
    sums[0] = s0 + partner_f(s0);
    sums[1] = s1 + partner_f(s1);
  } else if constexpr (MODE == kC8) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float s = (p[4 * i] + p[4 * i + 1]) + (p[4 * i + 2] + p[4 * i + 3]);
      sums[i] = s + partner_f(s);
    }
  } else {  // kC4: chunk 2i+h lives entirely in lane half h
#pragma unroll
    for (int i = 0; i < 4; ++i) sums[i] = (p[4 * i] + p[4 * i + 1]) + (p[4 * i + 2] + p[4 * i + 3]);
  }
}

template <int MODE>
constexpr int sums_per_lane() {
  return MODE >= kC32 ? 1 : MODE == kC16 ? 2 : 4;
}

struct RangeState {
  float mref[2];       // per row tile: reference (scaled log2 units)
  double zsum[2];      // per row tile: sum of the range's chunk sums
  float chunk_acc[2];  // kC32x with c > 32: running sum of the open chunk
  bool overflow;
};

// One 32-key subtile (range-relative keys rk0 .. rk0+31 of a range holding
// nkeys keys), read from LDS rows lrow0 .. lrow0+31.  FULL: all 32 keys valid
// (uniform; only a range's last subtile can be short).  PASS 0 and PASS 2:
// partial sums against st.mref.  PASS 1: exact range maximum only.
template <int D, int MODE, int PASS, bool FULL, bool QMEM = false>
__device__ __forceinline__ void process_subtile(const ScoreArgs& a, const bf16x8 (&qf)[2][D / 16],
                                                const uint16_t* lds, int lrow0, int rk0, int nkeys,
                                                float* part, int my_row0, RangeState& st,
                                                int g = 0) {
  const int lane = threadIdx.x & 63, half = lane >> 5;
  f32x16 acc[2];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[rt][v] = 0.f;
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    bf16x8 kf = *reinterpret_cast<const bf16x8*>(
        lds + SubtileLds<D>::offset(lrow0 + (lane & 31), 2 * ks + half));
    acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[0][ks], acc[0], 0, 0, 0);
    acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[1][ks], acc[1], 0, 0, 0);
  }
  // register v of this lane holds key rk0 + 8*(v/4) + 4*half + v%4
  const int nvalid = FULL ? kSub : min(kSub, nkeys - rk0);

  if (PASS == 1) {
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      float mx = -INFINITY;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int key = 8 * (v >> 2) + 4 * half + (v & 3);
        if (FULL || key < nvalid) mx = fmaxf(mx, acc[rt][v]);
      }
      mx = fmaxf(mx, partner_f(mx));
      st.mref[rt] = fmaxf(st.mref[rt], mx * a.c1);
    }
    return;
  }

  // p = exp2(c1*dot - mc); keys past the range's end contribute 0
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    const float nm = -st.mref[rt];
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const float e = __builtin_amdgcn_exp2f(fmaf(acc[rt][v], a.c1, nm));
      if constexpr (FULL) {
        acc[rt][v] = e;
      } else {
        const int key = 8 * (v >> 2) + 4 * half + (v & 3);
        acc[rt][v] = key < nvalid ? e : 0.f;
      }
    }
  }

  if constexpr (MODE >= kC32) {
    const bool closes = ((rk0 + kSub) % a.c == 0) || (rk0 + kSub >= nkeys);
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      float sum;
      chunk_sums<MODE>(acc[rt], &sum);
      st.chunk_acc[rt] += sum;
    }
    if (closes) {
      const int jl = rk0 / a.c;
      const int row = my_row0 + lane;  // lane l writes row tile l/32, row l%32
      const float mine = half ? st.chunk_acc[1] : st.chunk_acc[0];
      part[(int64_t)jl * a.ldp + row] = mine;
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        st.overflow |= !(st.chunk_acc[rt] <= kOverflowGuard);
        st.zsum[rt] += (double)st.chunk_acc[rt];
        st.chunk_acc[rt] = 0.f;
      }
    }
  } else {
    constexpr int kN = sums_per_lane<MODE>();
    constexpr int kChunk = MODE == kC4 ? 4 : MODE == kC8 ? 8 : 16;
    const int jl0 = rk0 / kChunk;  // first chunk of this subtile
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      float sums[kN];
      chunk_sums<MODE>(acc[rt], sums);
#pragma unroll
      for (int i = 0; i < kN; ++i) {
        st.overflow |= !(sums[i] <= kOverflowGuard);
        st.zsum[rt] += (double)sums[i];
      }
      if constexpr (MODE == kC4) {
        // lane half h holds chunks 2i+h of rows (row tile rt, row lane%32)
        const int row = my_row0 + rt * 32 + (lane & 31);
#pragma unroll
        for (int i = 0; i < kN; ++i) {
          const int key_first = 8 * i + 4 * half;
          if (FULL || key_first < nvalid) part[(int64_t)(jl0 + 2 * i + half) * a.ldp + row] = sums[i];
        }
      } else if (rt == half) {
        // both halves hold every sum: half h writes row tile h
        const int row = my_row0 + rt * 32 + (lane & 31);
#pragma unroll
        for (int i = 0; i < kN; ++i) {
          const int key_first = i * (kSub / kN);
          if (FULL || key_first < nvalid) part[(int64_t)(jl0 + i) * a.ldp + row] = sums[i];
        }
      }
    }
  }
}

// Common softmax reference of each row: the scaled maximum of its logits over
// the prefix's first 32 keys.  Every workgroup of a row computes the same value,
// so all key ranges of a row share one reference and the fold across ranges
// needs no rescaling (unless a range fell back to its exact maximum).
template <int D>
__device__ void row_reference(const ScoreArgs& a, int g, const bf16x8 (&qf)[2][D / 16],
                              uint16_t* lds, RangeState& st) {
  constexpr int kSegs = D / 8;
  constexpr int kPer = StageRegs<D>::kPer;
  const int lane = threadIdx.x & 63, half = lane >> 5;
  const int nkeys = (int)min<int64_t>(kSub, a.n);
  uint32_t voff[kPer], voff0[kPer];
#pragma unroll
  for (int p = 0; p < kPer; ++p) {
    const int idx = threadIdx.x + p * kWaves * 64;
    voff[p] = (uint32_t)(((int64_t)(idx / kSegs) * a.Hkv + g) * D + (idx % kSegs) * 8);
    voff0[p] = (uint32_t)(g * D + (idx % kSegs) * 8);
  }
  StageRegs<D> r;
  stage_load<D>(a.k, nkeys, voff, voff0, r);
  stage_store<D>(r, lds);
  __syncthreads();
  f32x16 acc[2];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[rt][v] = 0.f;
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    bf16x8 kf = *reinterpret_cast<const bf16x8*>(lds + SubtileLds<D>::offset(lane & 31, 2 * ks + half));
    acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[0][ks], acc[0], 0, 0, 0);
    acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[1][ks], acc[1], 0, 0, 0);
  }
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    float mx = -INFINITY;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int key = 8 * (v >> 2) + 4 * half + (v & 3);
      if (key < nkeys) mx = fmaxf(mx, acc[rt][v]);
    }
    mx = fmaxf(mx, partner_f(mx));
    st.mref[rt] = mx * a.c1;
  }
  __syncthreads();  // LDS is reused by the range
}

// ---- software-pipelined steady state (PASS 0, full 64-key stages) ----------
// A stage is four units (subtile 0/1 x row tile 0/1).  Each unit's 8 MFMAs are
// issued while the previous unit's softmax VALU work runs, in one basic block,
// and the last unit's VALU work is carried over the stage barrier into the next
// stage.  Scheduling-group hints ask the scheduler to alternate the two.

// All 16 MFMAs of one subtile (both row tiles share each K fragment).
template <int D>
__device__ __forceinline__ void mfma_subtile(const uint16_t* lds, int lrow0,
                                             const bf16x8 (&qf)[2][D / 16], f32x16 (&acc)[2]) {
  const int lane = threadIdx.x & 63, half = lane >> 5;
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[rt][v] = 0.f;
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    const bf16x8 kf = *reinterpret_cast<const bf16x8*>(
        lds + SubtileLds<D>::offset(lrow0 + (lane & 31), 2 * ks + half));
    acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[0][ks], acc[0], 0, 0, 0);
    acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[1][ks], acc[1], 0, 0, 0);
  }
}

// Softmax numerators, per-chunk sums, partial writes and z for one unit: row
// tile RT of a full 32-key subtile starting at range-relative key rk0.  Both
// lane halves hold the combined sums; each pair of lanes writes the same value
// to the same row (rows are padded, so no guard is needed).
template <int MODE, int RT>
__device__ __forceinline__ void valu_unit(const ScoreArgs& a, f32x16& acc, int rk0, float* part,
                                          int my_row0, RangeState& st) {
  const int lane = threadIdx.x & 63, half = lane >> 5;
  const float nm = -st.mref[RT];
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = __builtin_amdgcn_exp2f(fmaf(acc[v], a.c1, nm));
  constexpr int kN = sums_per_lane<MODE>();
  float sums[kN];
  chunk_sums<MODE>(acc, sums);
  const int row = my_row0 + RT * 32 + (lane & 31);
  if constexpr (MODE == kC32) {
    part[(int64_t)(rk0 >> 5) * a.ldp + row] = sums[0];
    st.overflow |= !(sums[0] <= kOverflowGuard);
    st.zsum[RT] += (double)sums[0];
  } else if constexpr (MODE == kC32x) {
    st.chunk_acc[RT] += sums[0];
    if ((rk0 + kSub) % a.c == 0) {  // uniform
      part[(int64_t)(rk0 / a.c) * a.ldp + row] = st.chunk_acc[RT];
      st.overflow |= !(st.chunk_acc[RT] <= kOverflowGuard);
      st.zsum[RT] += (double)st.chunk_acc[RT];
      st.chunk_acc[RT] = 0.f;
    }
  } else {
    constexpr int kChunk = MODE == kC4 ? 4 : MODE == kC8 ? 8 : 16;
    const int jl0 = rk0 / kChunk;
#pragma unroll
    for (int i = 0; i < kN; ++i) {
      st.overflow |= !(sums[i] <= kOverflowGuard);
      st.zsum[RT] += (double)sums[i];
      // kC4: lane half h holds chunks 2i+h; otherwise both halves hold chunk i
      const int jl = MODE == kC4 ? jl0 + 2 * i + half : jl0 + i;
      part[(int64_t)jl * a.ldp + row] = sums[i];
    }
  }
}

// Asks the scheduler to alternate the 16 MFMAs of a slot with VALU work.
__device__ __forceinline__ void interleave_hint() {
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
    __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);  // then VALU
  }
}

// One full 64-key stage as two slots.  Slot 0: MFMAs of subtile 0 with the
// VALU work of the subtile carried from the previous stage; slot 1: MFMAs of
// subtile 1 (into `carry`) with the VALU work of subtile 0.
template <int D, int MODE, bool CARRY>
__device__ __forceinline__ void fast_stage(const ScoreArgs& a, const bf16x8 (&qf)[2][D / 16],
                                           const uint16_t* cur, int rk0, float* part, int my_row0,
                                           RangeState& st, f32x16 (&carry)[2], int& carry_rk) {
  f32x16 acc[2];
  __builtin_amdgcn_sched_barrier(0);
  mfma_subtile<D>(cur, 0, qf, acc);
  if constexpr (CARRY) {
    valu_unit<MODE, 0>(a, carry[0], carry_rk, part, my_row0, st);
    valu_unit<MODE, 1>(a, carry[1], carry_rk, part, my_row0, st);
    interleave_hint();
  }
  __builtin_amdgcn_sched_barrier(0);
  mfma_subtile<D>(cur, kSub, qf, carry);
  valu_unit<MODE, 0>(a, acc[0], rk0, part, my_row0, st);
  valu_unit<MODE, 1>(a, acc[1], rk0, part, my_row0, st);
  interleave_hint();
  __builtin_amdgcn_sched_barrier(0);
  carry_rk = rk0 + kSub;
}

// PASS 0 over the range: pipelined full stages, then the short tail stage (if
// any) through process_subtile.
template <int D, int MODE>
__device__ bool run_range_fast(const ScoreArgs& a, int g, int range, int row0,
                               const bf16x8 (&qf)[2][D / 16], uint16_t* lds, RangeState& st) {
  constexpr int kSegs = D / 8;
  constexpr int kPer = StageRegs<D>::kPer;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5;
  const int64_t kbeg = (int64_t)range * a.key_range;
  const int nkeys = (int)(min<int64_t>(kbeg + a.key_range, a.n) - kbeg);
  const int nstage = (nkeys + kStage - 1) / kStage;
  const int nfull = nkeys / kStage;
  const int my_row0 = row0 + wave * kWaveRows;
  st.overflow = false;
  st.chunk_acc[0] = st.chunk_acc[1] = 0.f;
  st.zsum[0] = st.zsum[1] = 0.0;
  float* part = a.part + ((int64_t)(g * a.n_ranges + range) * a.cpr) * a.ldp;

  uint32_t voff[kPer], voff0[kPer];
#pragma unroll
  for (int p = 0; p < kPer; ++p) {
    const int idx = threadIdx.x + p * kWaves * 64;
    const int key = idx / kSegs, seg = idx % kSegs;
    voff[p] = (uint32_t)(((int64_t)key * a.Hkv + g) * D + seg * 8);
    voff0[p] = (uint32_t)(g * D + seg * 8);
  }
  const int64_t stage_elems = (int64_t)kStage * a.Hkv * D;
  const uint16_t* kbase = a.k + kbeg * a.Hkv * D;

  StageRegs<D> r;
  stage_load<D>(kbase, nkeys, voff, voff0, r);
  stage_store<D>(r, lds);
  __syncthreads();
  f32x16 carry[2];
  int carry_rk = 0;
  for (int s = 0; s < nfull; ++s) {
    const int rk0 = s * kStage;
    if (s + 1 < nstage) stage_load<D>(kbase + (s + 1) * stage_elems, nkeys - rk0 - kStage, voff, voff0, r);
    const uint16_t* cur = lds + (s & 1) * kStage * D;
    if (s == 0)
      fast_stage<D, MODE, false>(a, qf, cur, rk0, part, my_row0, st, carry, carry_rk);
    else
      fast_stage<D, MODE, true>(a, qf, cur, rk0, part, my_row0, st, carry, carry_rk);
    if (s + 1 < nstage) stage_store<D>(r, lds + ((s + 1) & 1) * kStage * D);
    __syncthreads();
  }
  if (nfull > 0) {
    valu_unit<MODE, 0>(a, carry[0], carry_rk, part, my_row0, st);
    valu_unit<MODE, 1>(a, carry[1], carry_rk, part, my_row0, st);
  }
  if (nfull < nstage) {  // short last stage
    const int rk0 = nfull * kStage;
    const uint16_t* cur = lds + (nfull & 1) * kStage * D;
    process_subtile<D, MODE, 0, false>(a, qf, cur, 0, rk0, nkeys, part, my_row0, st);
    if (rk0 + kSub < nkeys)
      process_subtile<D, MODE, 0, false>(a, qf, cur, kSub, rk0 + kSub, nkeys, part, my_row0, st);
  }
  if constexpr (MODE == kC4) {
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      const double o = partner_d(st.zsum[rt]);
      st.zsum[rt] = half ? (o + st.zsum[rt]) : (st.zsum[rt] + o);
    }
  }
  return st.overflow;
}

// Processes the workgroup's key range once (see process_subtile for PASS); used
// by the exact fallback kernel.
template <int D, int MODE, int PASS>
__device__ bool run_range(const ScoreArgs& a, int g, int range, int row0,
                          const bf16x8 (&qf)[2][D / 16], uint16_t* lds, RangeState& st) {
  constexpr int kSegs = D / 8;
  constexpr int kPer = StageRegs<D>::kPer;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5;
  const int64_t kbeg = (int64_t)range * a.key_range;
  const int nkeys = (int)(min<int64_t>(kbeg + a.key_range, a.n) - kbeg);
  const int nstage = (nkeys + kStage - 1) / kStage;
  const int my_row0 = row0 + wave * kWaveRows;
  st.overflow = false;
  st.chunk_acc[0] = st.chunk_acc[1] = 0.f;
  if (PASS != 1) st.zsum[0] = st.zsum[1] = 0.0;
  if (PASS == 1) st.mref[0] = st.mref[1] = -INFINITY;
  float* part = a.part + ((int64_t)(g * a.n_ranges + range) * a.cpr) * a.ldp;

  // per-thread element offsets of its pieces inside a stage (and of the stage's
  // first row, read in place of rows past the range end)
  uint32_t voff[kPer], voff0[kPer];
#pragma unroll
  for (int p = 0; p < kPer; ++p) {
    const int idx = threadIdx.x + p * kWaves * 64;
    const int key = idx / kSegs, seg = idx % kSegs;
    voff[p] = (uint32_t)(((int64_t)key * a.Hkv + g) * D + seg * 8);
    voff0[p] = (uint32_t)(g * D + seg * 8);
  }
  const int64_t stage_elems = (int64_t)kStage * a.Hkv * D;
  const uint16_t* kbase = a.k + kbeg * a.Hkv * D;

  StageRegs<D> r;
  stage_load<D>(kbase, nkeys, voff, voff0, r);
  stage_store<D>(r, lds);
  __syncthreads();
  for (int s = 0; s < nstage; ++s) {
    const int rk0 = s * kStage;
    if (s + 1 < nstage) stage_load<D>(kbase + (s + 1) * stage_elems, nkeys - rk0 - kStage, voff, voff0, r);
    const uint16_t* cur = lds + (s & 1) * kStage * D;
    if (rk0 + kStage <= nkeys) {
      process_subtile<D, MODE, PASS, true>(a, qf, cur, 0, rk0, nkeys, part, my_row0, st);
      process_subtile<D, MODE, PASS, true>(a, qf, cur, kSub, rk0 + kSub, nkeys, part, my_row0, st);
    } else {
      process_subtile<D, MODE, PASS, false>(a, qf, cur, 0, rk0, nkeys, part, my_row0, st);
      if (rk0 + kSub < nkeys)
        process_subtile<D, MODE, PASS, false>(a, qf, cur, kSub, rk0 + kSub, nkeys, part, my_row0, st);
    }
    if (s + 1 < nstage) stage_store<D>(r, lds + ((s + 1) & 1) * kStage * D);
    __syncthreads();
  }
  if constexpr (MODE == kC4) {
    // each half summed different chunks: combine in a fixed order (half 0 + half 1)
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      const double o = partner_d(st.zsum[rt]);
      st.zsum[rt] = half ? (o + st.zsum[rt]) : (st.zsum[rt] + o);
    }
  }
  return st.overflow;
}

// Q^T fragments of the workgroup's rows: B operand, lane l holds row l%32 of a
// row tile and d = 16*ks + 8*half .. +7 (zero past R).
template <int D>
__device__ __forceinline__ void load_q(const ScoreArgs& a, int g, int row0, bf16x8 (&qf)[2][D / 16]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5;
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    const int row = row0 + wave * kWaveRows + rt * 32 + (lane & 31);
    const bool ok = row < a.R;
    const int t = ok ? row / a.G : 0, hi = ok ? row % a.G : 0;
    const uint16_t* src = a.q + ((int64_t)t * a.Hq + (int64_t)g * a.G + hi) * D + 8 * half;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      u32x4 v = *reinterpret_cast<const u32x4*>(src + 16 * ks);
      if (!ok) v = u32x4{0u, 0u, 0u, 0u};
      qf[rt][ks] = *reinterpret_cast<bf16x8*>(&v);
    }
  }
}

__device__ __forceinline__ void store_stats(const ScoreArgs& a, int g, int range, int row0,
                                            const RangeState& st) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5;
  const int row = row0 + wave * kWaveRows + lane;  // lane l reports row tile l/32
  if (row < a.R) {
    const int64_t o = (int64_t)(g * a.n_ranges + range) * a.R + row;
    a.mc[o] = half ? st.mref[1] : st.mref[0];
    a.z[o] = half ? st.zsum[1] : st.zsum[0];
  }
}

// Main pass: every (KV head, key range, 256-row block) workgroup, pipelined,
// against the rows' common reference.  Records in flags[L] whether a chunk sum
// of its range overflowed (then the fallback kernel redoes the range).
template <int D, int MODE>
__global__ __launch_bounds__(kWaves * 64, 2) void score_bf16_kernel(ScoreArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * kStage * D];
  const uint32_t L = xcd_remap(blockIdx.x, a.nblocks_padded);
  if (L >= a.nblocks) return;
  const int rb = (int)(L % a.n_row_blocks);
  const int range = (int)((L / a.n_row_blocks) % a.n_ranges);
  const int g = (int)(L / ((uint32_t)a.n_row_blocks * a.n_ranges));
  const int row0 = rb * kBlockRows;
  bf16x8 qf[2][D / 16];
  load_q<D>(a, g, row0, qf);
  RangeState st;
  row_reference<D>(a, g, qf, lds, st);
  const bool of = run_range_fast<D, MODE>(a, g, range, row0, qf, lds, st);
  const int any_of = __syncthreads_or(of ? 1 : 0);
  if (threadIdx.x == 0) a.flags[L] = any_of;
  store_stats(a, g, range, row0, st);
}

// Exact fallback, almost always a no-op: a grid-stride loop over the main
// pass's workgroups; a flagged range is recomputed against its own exact
// maximum (first pass: maximum only, second pass: partial sums and z).
template <int D, int MODE>
__global__ __launch_bounds__(kWaves * 64, 2) void score_fallback_kernel(ScoreArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * kStage * D];
  // all threads scan this block's share of the flags at once; nothing to do is
  // the common case
  int mine = 0;
  for (uint32_t L = blockIdx.x + gridDim.x * threadIdx.x; L < a.nblocks; L += gridDim.x * blockDim.x)
    mine |= a.flags[L];
  if (!__syncthreads_or(mine)) return;
  for (uint32_t L = blockIdx.x; L < a.nblocks; L += gridDim.x) {
    if (!a.flags[L]) continue;  // uniform
    const int rb = (int)(L % a.n_row_blocks);
    const int range = (int)((L / a.n_row_blocks) % a.n_ranges);
    const int g = (int)(L / ((uint32_t)a.n_row_blocks * a.n_ranges));
    const int row0 = rb * kBlockRows;
    bf16x8 qf[2][D / 16];
    load_q<D>(a, g, row0, qf);
    RangeState st;
    run_range<D, MODE, 1>(a, g, range, row0, qf, lds, st);
    run_range<D, MODE, 2>(a, g, range, row0, qf, lds, st);
    store_stats(a, g, range, row0, st);
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// fp32 kernel (v_mfma_f32_32x32x2_f32), same structure without LDS staging:
// K fragments are read straight from global memory (the fp32 workloads are
// small).  One wave per workgroup, 64 rows.
// ---------------------------------------------------------------------------
struct ScoreArgsF32 {
  const float* q;
  const float* k;
  float* part;
  float* mc;
  double* z;
  int64_t n;
  int S, Hq, Hkv, G, R, ldp, c, key_range, n_ranges, cpr, n_row_blocks;
  float c1;
  uint32_t nblocks;
};

template <int D, int MODE, int PASS>
__device__ bool run_range_f32(const ScoreArgsF32& a, int g, int range, int row0,
                              const float (&qf)[2][D / 2], float (&mref)[2], double (&zsum)[2]) {
  const int lane = threadIdx.x & 63, half = lane >> 5;
  const int64_t kbeg = (int64_t)range * a.key_range;
  const int64_t kend = min<int64_t>(kbeg + a.key_range, a.n);
  const int nsub = (int)((kend - kbeg + kSub - 1) / kSub);
  bool overflow = false;
  float chunk_acc[2] = {0.f, 0.f};
  if (PASS != 1) { zsum[0] = 0.0; zsum[1] = 0.0; }
  if (PASS == 1) { mref[0] = -INFINITY; mref[1] = -INFINITY; }
  float* part = a.part + ((int64_t)(g * a.n_ranges + range) * a.cpr) * a.ldp;
  for (int s = 0; s < nsub; ++s) {
    const int64_t key0 = kbeg + (int64_t)s * kSub;
    const int nvalid = (int)min<int64_t>(kSub, kend - key0);
    const int64_t mykey = key0 + (lane & 31);
    const float* krow = a.k + (min<int64_t>(mykey, a.n - 1) * a.Hkv + g) * D;
    f32x16 acc[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[rt][v] = 0.f;
#pragma unroll
    for (int ks = 0; ks < D / 2; ++ks) {
      float kf = krow[2 * ks + half];
      acc[0] = __builtin_amdgcn_mfma_f32_32x32x2f32(kf, qf[0][ks], acc[0], 0, 0, 0);
      acc[1] = __builtin_amdgcn_mfma_f32_32x32x2f32(kf, qf[1][ks], acc[1], 0, 0, 0);
    }
    if (PASS == 1 || (PASS == 0 && s == 0)) {
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        float mx = -INFINITY;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          int key = 8 * (v >> 2) + 4 * half + (v & 3);
          if (key < nvalid) mx = fmaxf(mx, acc[rt][v]);
        }
        mx = fmaxf(mx, partner_f(mx));
        if (PASS == 1)
          mref[rt] = fmaxf(mref[rt], mx * a.c1);
        else
          mref[rt] = mx * a.c1;
      }
    }
    if (PASS == 1) continue;
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      const float nm = -mref[rt];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        int key = 8 * (v >> 2) + 4 * half + (v & 3);
        float e = __builtin_amdgcn_exp2f(fmaf(acc[rt][v], a.c1, nm));
        acc[rt][v] = key < nvalid ? e : 0.f;
      }
    }
    if constexpr (MODE >= kC32) {
      const int64_t chunk = key0 / a.c;
      const bool closes = ((key0 + kSub) % a.c == 0) || (s == nsub - 1);
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        float sum;
        chunk_sums<MODE>(acc[rt], &sum);
        chunk_acc[rt] += sum;
      }
      if (closes) {
        const int jl = (int)(chunk - kbeg / a.c);
        const int row = row0 + lane;
        float mine = half ? chunk_acc[1] : chunk_acc[0];
        if (row < a.R) part[(int64_t)jl * a.ldp + row] = mine;
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          overflow |= !(chunk_acc[rt] <= kOverflowGuard);
          zsum[rt] += (double)chunk_acc[rt];
          chunk_acc[rt] = 0.f;
        }
      }
    } else {
      constexpr int kN = sums_per_lane<MODE>();
      const int jl0 = (int)((key0 - kbeg) / a.c);
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        float sums[kN];
        chunk_sums<MODE>(acc[rt], sums);
#pragma unroll
        for (int i = 0; i < kN; ++i) {
          overflow |= !(sums[i] <= kOverflowGuard);
          zsum[rt] += (double)sums[i];
        }
        if constexpr (MODE == kC4) {
          const int row = row0 + rt * 32 + (lane & 31);
#pragma unroll
          for (int i = 0; i < kN; ++i) {
            int jl = jl0 + 2 * i + half;
            int key_first = 8 * i + 4 * half;
            if (row < a.R && key_first < nvalid) part[(int64_t)jl * a.ldp + row] = sums[i];
          }
        } else if (rt == half) {
          const int row = row0 + rt * 32 + (lane & 31);
#pragma unroll
          for (int i = 0; i < kN; ++i) {
            int key_first = i * (kSub / kN);
            if (row < a.R && key_first < nvalid) part[(int64_t)(jl0 + i) * a.ldp + row] = sums[i];
          }
        }
      }
    }
  }
  if constexpr (MODE == kC4) {
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      double o = partner_d(zsum[rt]);
      zsum[rt] = half ? (o + zsum[rt]) : (zsum[rt] + o);
    }
  }
  return overflow;
}

template <int D, int MODE>
__global__ __launch_bounds__(64) void score_f32_kernel(ScoreArgsF32 a) {
  const uint32_t L = blockIdx.x;
  if (L >= a.nblocks) return;
  const int rb = (int)(L % a.n_row_blocks);
  const int range = (int)((L / a.n_row_blocks) % a.n_ranges);
  const int g = (int)(L / ((uint32_t)a.n_row_blocks * a.n_ranges));
  const int lane = threadIdx.x & 63, half = lane >> 5;
  const int row0 = rb * kWaveRows;
  float qf[2][D / 2];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    const int row = row0 + rt * 32 + (lane & 31);
    const bool ok = row < a.R;
    const int t = ok ? row / a.G : 0, hi = ok ? row % a.G : 0;
    const float* src = a.q + ((int64_t)t * a.Hq + (int64_t)g * a.G + hi) * D + half;
#pragma unroll
    for (int ks = 0; ks < D / 2; ++ks) qf[rt][ks] = ok ? src[2 * ks] : 0.f;
  }
  float mref[2];
  double zsum[2];
  bool of = run_range_f32<D, MODE, 0>(a, g, range, row0, qf, mref, zsum);
  // one wave: the decision is wave-uniform via a ballot
  if (__any(of)) {
    run_range_f32<D, MODE, 1>(a, g, range, row0, qf, mref, zsum);
    run_range_f32<D, MODE, 2>(a, g, range, row0, qf, mref, zsum);
  }
  const int row = row0 + lane;
  if (row < a.R) {
    const int64_t o = (int64_t)(g * a.n_ranges + range) * a.R + row;
    a.mc[o] = half ? mref[1] : mref[0];
    a.z[o] = half ? zsum[1] : zsum[0];
  }
}

// ---------------------------------------------------------------------------
// finalize
// ---------------------------------------------------------------------------
// F1: per (g, row): Mc = max over ranges of mc, Z = sum over ranges of
// exp2(mc - Mc) z, and the z slot of every range is overwritten with
// w = exp2(mc - Mc) / Z (fp64).  All ranges normally share one reference (then
// every factor exp2(0) = 1 is exact and skipped); a range that fell back to its
// own maximum is rescaled here.  A workgroup serves 32 rows (coalesced) with 8
// lanes per row splitting the ranges; partial results are combined through LDS
// in lane order.
constexpr int kNormRows = 32;
constexpr int kNormLanes = 8;

__device__ __forceinline__ double range_factor(float mc, float M) {
  return mc == M ? 1.0 : exp2((double)mc - (double)M);
}

__global__ __launch_bounds__(kNormRows * kNormLanes) void row_norm_kernel(
    const float* __restrict__ mc, double* __restrict__ z, int Hkv, int R, int NR) {
  __shared__ float smax[kNormLanes][kNormRows];
  __shared__ double ssum[kNormLanes][kNormRows];
  const int rl = threadIdx.x % kNormRows, q = threadIdx.x / kNormRows;
  const int blocks_per_head = (R + kNormRows - 1) / kNormRows;
  const int g = blockIdx.x / blocks_per_head;
  const int row = (blockIdx.x % blocks_per_head) * kNormRows + rl;
  const bool ok = row < R;
  const int64_t base = (int64_t)g * NR * R + row;
  float M = -INFINITY;
  if (ok)
    for (int r = q; r < NR; r += kNormLanes) M = fmaxf(M, mc[base + (int64_t)r * R]);
  smax[q][rl] = M;
  __syncthreads();
  M = smax[0][rl];
  for (int i = 1; i < kNormLanes; ++i) M = fmaxf(M, smax[i][rl]);
  double Z = 0.0;
  if (ok)
    for (int r = q; r < NR; r += kNormLanes)
      Z += range_factor(mc[base + (int64_t)r * R], M) * z[base + (int64_t)r * R];
  ssum[q][rl] = Z;
  __syncthreads();
  Z = ssum[0][rl];
  for (int i = 1; i < kNormLanes; ++i) Z += ssum[i][rl];
  if (!ok) return;
  const double inv = 1.0 / Z;
  for (int r = q; r < NR; r += kNormLanes)
    z[base + (int64_t)r * R] = range_factor(mc[base + (int64_t)r * R], M) * inv;
}

// F2: A_j = sum over KV heads g (in order) of sum over rows r of
// w[g][range(j)][r] * P[g][range(j)][jl][r], in fp64.  One workgroup of 256
// threads per chunk: thread i takes rows i, i+256, ... of every head in order,
// then a fixed tree over LDS reduces the 256 partial sums.
constexpr int kReduceThreads = 256;

__global__ __launch_bounds__(kReduceThreads) void chunk_reduce_kernel(
    const float* __restrict__ part, const double* __restrict__ w, double* __restrict__ A, int Hkv,
    int R, int ldp, int NR, int cpr) {
  __shared__ double red[kReduceThreads];
  const int64_t j = blockIdx.x;
  const int tid = threadIdx.x;
  const int range = (int)(j / cpr), jl = (int)(j % cpr);
  double s = 0.0;
  for (int g = 0; g < Hkv; ++g) {
    const float* p = part + (((int64_t)g * NR + range) * cpr + jl) * ldp;
    const double* wr = w + ((int64_t)g * NR + range) * R;
    for (int r = tid; r < R; r += kReduceThreads) s += (double)p[r] * wr[r];
  }
  red[tid] = s;
  __syncthreads();
#pragma unroll
  for (int width = kReduceThreads / 2; width >= 64; width >>= 1) {
    if (tid < width) red[tid] += red[tid + width];
    __syncthreads();
  }
  if (tid < 64) {
    s = red[tid];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off);
    if (tid == 0) A[j] = s;
  }
}

int chunk_mode(int c) {
  if (c == 4) return kC4;
  if (c == 8) return kC8;
  if (c == 16) return kC16;
  if (c == 32) return kC32;
  if (c % 32 == 0) return kC32x;
  return -1;
}

}  // namespace

ScorePlan make_score_plan(const ckv_dims* d) {
  ScorePlan p{};
  const int G = d->n_q_heads / d->n_kv_heads;
  p.m = ceil_div(d->n_prefix, d->chunk_size);
  p.rows = G * d->n_suffix;
  const int unit = d->chunk_size % 32 == 0 ? d->chunk_size : 32;  // lcm(32, c) for supported c
  const bool f32 = d->dtype == CKV_DTYPE_F32;
  const int64_t row_blocks = ceil_div(p.rows, f32 ? kWaveRows : kBlockRows);
  // Longer key ranges amortise each workgroup's fixed work (Q tile, row
  // reference, statistics) and shrink the per-range partials that the
  // normalisation pass reads; grow the range while the grid keeps at least
  // 1.5 workgroups per CU.
  int64_t kr = unit * ceil_div(256, unit);
  while (kr * 2 <= 4096 && (int64_t)d->n_kv_heads * row_blocks * ceil_div(d->n_prefix, kr * 2) >= 384)
    kr *= 2;
  p.key_range = (int32_t)kr;
  p.n_ranges = (int32_t)ceil_div(d->n_prefix, kr);
  p.cpr = (int32_t)(kr / d->chunk_size);
  p.ldp = (int32_t)align_up(p.rows, kBlockRows);
  const size_t R = (size_t)p.rows, H = (size_t)d->n_kv_heads, NR = (size_t)p.n_ranges;
  size_t off = 0;
  p.off_part = off;
  off = align_up(off + H * NR * p.cpr * (size_t)p.ldp * sizeof(float), 256);
  p.off_mc = off;
  off = align_up(off + H * NR * R * sizeof(float), 256);
  p.off_z = off;
  off = align_up(off + H * NR * R * sizeof(double), 256);
  p.off_flags = off;
  off = align_up(off + H * NR * (size_t)ceil_div(p.rows, kBlockRows) * sizeof(int), 256);
  p.bytes = off;
  return p;
}

ckv_status launch_score(const ckv_dims* d, const void* q, const void* k, double* scores, void* ws,
                        size_t ws_bytes, hipStream_t st, hipEvent_t after_main) {
  const ScorePlan p = make_score_plan(d);
  if (ws_bytes < p.bytes) CKV_FAIL(CKV_EINVAL, "score workspace too small: %zu < %zu", ws_bytes, p.bytes);
  const int mode = chunk_mode(d->chunk_size);
  char* base = static_cast<char*>(ws);
  float* part = reinterpret_cast<float*>(base + p.off_part);
  float* mc = reinterpret_cast<float*>(base + p.off_mc);
  double* z = reinterpret_cast<double*>(base + p.off_z);
  const int G = d->n_q_heads / d->n_kv_heads;
  const float c1 = resolve_scale(d) * 1.4426950408889634f;

  if (d->dtype == CKV_DTYPE_BF16) {
    ScoreArgs a;
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.part = part; a.mc = mc; a.z = z;
    a.flags = reinterpret_cast<int*>(base + p.off_flags);
    a.n = d->n_prefix; a.S = d->n_suffix; a.Hq = d->n_q_heads; a.Hkv = d->n_kv_heads; a.G = G;
    a.R = p.rows; a.ldp = p.ldp; a.c = d->chunk_size; a.key_range = p.key_range;
    a.n_ranges = p.n_ranges; a.cpr = p.cpr; a.n_row_blocks = (int)ceil_div(p.rows, kBlockRows);
    a.c1 = c1;
    a.nblocks = (uint32_t)((int64_t)a.Hkv * a.n_ranges * a.n_row_blocks);
    a.nblocks_padded = (uint32_t)align_up(a.nblocks, 8);
    dim3 grid(a.nblocks_padded), block(kWaves * 64);
#define CKV_SCORE_LAUNCH(DD, MM)                                                        \
  do {                                                                                  \
    hipLaunchKernelGGL((score_bf16_kernel<DD, MM>), grid, block, 0, st, a);             \
    hipLaunchKernelGGL((score_fallback_kernel<DD, MM>), dim3(kFallbackBlocks), block, 0, st, a); \
  } while (0)
    if (d->head_dim == 128) {
      switch (mode) {
        case kC4: CKV_SCORE_LAUNCH(128, kC4); break;
        case kC8: CKV_SCORE_LAUNCH(128, kC8); break;
        case kC16: CKV_SCORE_LAUNCH(128, kC16); break;
        case kC32: CKV_SCORE_LAUNCH(128, kC32); break;
        default: CKV_SCORE_LAUNCH(128, kC32x); break;
      }
    } else {
      switch (mode) {
        case kC4: CKV_SCORE_LAUNCH(64, kC4); break;
        case kC8: CKV_SCORE_LAUNCH(64, kC8); break;
        case kC16: CKV_SCORE_LAUNCH(64, kC16); break;
        case kC32: CKV_SCORE_LAUNCH(64, kC32); break;
        default: CKV_SCORE_LAUNCH(64, kC32x); break;
      }
    }
#undef CKV_SCORE_LAUNCH
  } else {
    ScoreArgsF32 a;
    a.q = static_cast<const float*>(q);
    a.k = static_cast<const float*>(k);
    a.part = part; a.mc = mc; a.z = z;
    a.n = d->n_prefix; a.S = d->n_suffix; a.Hq = d->n_q_heads; a.Hkv = d->n_kv_heads; a.G = G;
    a.R = p.rows; a.ldp = p.ldp; a.c = d->chunk_size; a.key_range = p.key_range;
    a.n_ranges = p.n_ranges; a.cpr = p.cpr; a.n_row_blocks = (int)ceil_div(p.rows, kWaveRows);
    a.c1 = c1;
    a.nblocks = (uint32_t)((int64_t)a.Hkv * a.n_ranges * a.n_row_blocks);
    dim3 grid(a.nblocks), block(64);
    switch (mode) {
      case kC4: hipLaunchKernelGGL((score_f32_kernel<64, kC4>), grid, block, 0, st, a); break;
      case kC8: hipLaunchKernelGGL((score_f32_kernel<64, kC8>), grid, block, 0, st, a); break;
      case kC16: hipLaunchKernelGGL((score_f32_kernel<64, kC16>), grid, block, 0, st, a); break;
      case kC32: hipLaunchKernelGGL((score_f32_kernel<64, kC32>), grid, block, 0, st, a); break;
      default: hipLaunchKernelGGL((score_f32_kernel<64, kC32x>), grid, block, 0, st, a); break;
    }
  }
  CKV_HIP(hipGetLastError());
  if (after_main) CKV_HIP(hipEventRecord(after_main, st));
  const int norm_blocks = d->n_kv_heads * (int)ceil_div(p.rows, kNormRows);
  hipLaunchKernelGGL(row_norm_kernel, dim3(norm_blocks), dim3(kNormRows * kNormLanes), 0, st, mc,
                     z, d->n_kv_heads, p.rows, p.n_ranges);
  CKV_HIP(hipGetLastError());
  hipLaunchKernelGGL(chunk_reduce_kernel, dim3((unsigned)p.m), dim3(kReduceThreads), 0, st, part,
                     z, scores, d->n_kv_heads, p.rows, p.ldp, p.n_ranges, p.cpr);
  CKV_HIP(hipGetLastError());
  return CKV_OK;
}

}  // namespace ckv
