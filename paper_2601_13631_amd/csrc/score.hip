// score.hip -- chunk scoring (Sec. 4.4, Eq. 1) for gfx950.
//
// A_j = sum over rows r=(t,h) of sum_{i in chunk j} p_{r,i},
// p_{r,i} = softmax_i(sm_scale * q_r . k_i) over the n prefix keys.
//
// Work split.  Rows of one KV head g are r = t*G + i (query t, head g*G+i),
// grouped in blocks of 256 rows (4 waves x 64).  Each (KV head, row block) pair
// spans the whole key axis, cut into 256-key items; the items are dealt out in
// equal contiguous runs to a fixed grid of workgroups, so every workgroup (and
// CU) does the same work.  The items of one workgroup that share a row block
// form a segment.  Each wave keeps its 64 query rows in registers as the B
// operand of bf16 MFMA 32x32x16 and streams the segment's keys through LDS in
// 64-key stages of two 32-key subtiles, computing S^T = K Q^T so that every
// lane holds one query row and 16 of the 32 keys of a subtile (its partner lane
// l^32 the other 16).
//
// Softmax without a second pass.  A segment takes as each row's reference mc
// the scaled maximum of its logits over the segment's first 32 keys, rounded
// up to a whole number, and accumulates, per chunk, P = sum exp2(c1*dot - mc)
// (c1 = sm_scale*log2 e) in fp32 over at most one chunk, plus z = sum of the
// segment's chunk sums in fp64.  A fold kernel combines the segments of a row
// in fp64: M = max mc, Z = sum exp2(mc - M) z, w = exp2(mc - M)/Z (exact
// powers of two), and a reduction forms A_j = sum_r w P.  The result is exact
// in real arithmetic for any reference; the reference only has to keep exp2
// finite.  If a segment's z leaves the guard (some chunk sum is above it or not
// finite) the fold kernel first recomputes that segment against its own exact
// maximum (two passes), so the fast path never trades correctness for speed.
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

enum ChunkMode { kC4 = 0, kC8 = 1, kC16 = 2, kC32 = 3, kC32x = 4 };  // kC32x: c = 64, 96, ...

__device__ __forceinline__ float partner_f(float x) {
  // value of the same register in lane l^32
  int v = __float_as_int(x);
  auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return __int_as_float(threadIdx.x & 32 ? r[0] : r[1]);
}

// x + (x of lane l^32), the same value in both lanes of the pair.  The swap
// leaves (own, partner) in lanes 0..31 and (partner, own) in lanes 32..63, and
// fp32 addition is commutative, so no lane select is needed.
__device__ __forceinline__ float pair_sum(float x) {
  int v = __float_as_int(x);
  auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return __int_as_float(r[0]) + __int_as_float(r[1]);
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
// LDS stage: key rows of D bf16 padded by one 16-byte segment, so that the MFMA
// operand reads (consecutive lanes = consecutive keys, same segment) start 4
// banks apart and every 16-lane group covers all 64 banks once.  The padding
// keeps each fragment's address a compile-time offset from one base register.
template <int D>
struct SubtileLds {
  static constexpr int kRow = D + 8;  // elements per key row
  __device__ static int offset(int key, int seg) {  // in bf16 elements
    return key * kRow + seg * 8;
  }
};

struct ScoreArgs {
  const uint16_t* q;   // [S][Hq][D] bf16 bits
  const uint16_t* k;   // [n][Hkv][D]
  float* part;         // [Hkv][m_pad][ldp]
  float* mc;           // [Hkv*RB][NS][rpb]
  double* z;           // [Hkv*RB][NS][rpb]
  int* flags;          // [Hkv*RB][NS]: the segment overflowed in the main pass
  int64_t n, m_pad;    // keys; chunk slots per KV head (U*UK/c)
  int S, Hq, Hkv, G, R, c;
  float c1;            // sm_scale * log2(e)
  ScoreWork w;
  uint32_t nwg, nwg_padded;  // Hkv*RB*NS workgroups (the flags are indexed by workgroup)
  unsigned long long* tstamp;  // optional [nwg][2]: each workgroup's start and end (realtime clock)
};

constexpr int kStage = 64;  // keys per LDS stage: two 32-key subtiles

// The next stage's K rows are fetched into registers while the current stage is
// consumed from LDS, then written to the other LDS buffer: one barrier per stage.
// Loads are unconditional (rows past the segment end read the stage's first row
// and are zeroed when stored), so the compiler never has to wait on them early.
template <int D>
struct StageRegs {
  static constexpr int kPer = kStage * (D / 8) / (kWaves * 64);  // 16-byte loads per thread
  u32x4 v[kPer];
  uint32_t valid;  // bit p: piece p is inside the segment
};

// Byte offsets of a thread's pieces inside a stage (boff) and of the same
// segment of the stage's first key (boff0).
template <int D>
struct StageOffsets {
  uint32_t boff[StageRegs<D>::kPer], boff0[StageRegs<D>::kPer];
  __device__ StageOffsets(int Hkv, int g) {
    constexpr int kSegs = D / 8;
#pragma unroll
    for (int p = 0; p < StageRegs<D>::kPer; ++p) {
      const int idx = threadIdx.x + p * kWaves * 64;
      const int key = idx / kSegs, seg = idx % kSegs;
      boff[p] = (uint32_t)((((int64_t)key * Hkv + g) * D + seg * 8) * 2);
      boff0[p] = (uint32_t)((g * D + seg * 8) * 2);
    }
  }
};

// A stage that lies wholly inside the segment: plain loads from a uniform base.
template <int D>
__device__ __forceinline__ void stage_load_full(const uint16_t* kstage, const StageOffsets<D>& o,
                                                StageRegs<D>& r) {
  const char* base = reinterpret_cast<const char*>(kstage);
#pragma unroll
  for (int p = 0; p < StageRegs<D>::kPer; ++p)
    r.v[p] = *reinterpret_cast<const u32x4*>(base + o.boff[p]);
}

// A stage that may run past the segment end: rows past it read the stage's first
// row (always valid) and are zeroed by stage_store.
template <int D>
__device__ __forceinline__ void stage_load(const uint16_t* kstage, int64_t keys_left,
                                           const StageOffsets<D>& o, StageRegs<D>& r) {
  constexpr int kSegs = D / 8;
  const char* base = reinterpret_cast<const char*>(kstage);
  r.valid = 0;
#pragma unroll
  for (int p = 0; p < StageRegs<D>::kPer; ++p) {
    const int key = (threadIdx.x + p * kWaves * 64) / kSegs;
    const bool ok = key < keys_left;
    r.valid |= (ok ? 1u : 0u) << p;
    r.v[p] = *reinterpret_cast<const u32x4*>(base + (ok ? o.boff[p] : o.boff0[p]));
  }
}

template <int D, bool FULL>
__device__ __forceinline__ void stage_store(const StageRegs<D>& r, uint16_t* lds) {
  constexpr int kSegs = D / 8;
#pragma unroll
  for (int p = 0; p < StageRegs<D>::kPer; ++p) {
    const int idx = threadIdx.x + p * kWaves * 64;
    u32x4 v = r.v[p];
    if (!FULL && !((r.valid >> p) & 1u)) v = u32x4{0u, 0u, 0u, 0u};
    *reinterpret_cast<u32x4*>(lds + SubtileLds<D>::offset(idx / kSegs, idx % kSegs)) = v;
  }
}

// Per-chunk sums of one subtile for one row tile, combined across the lane pair.
// Fills sums[] (how many depends on the mode) in the order of chunk index.
template <int MODE>
__device__ __forceinline__ void chunk_sums(const f32x16& p, float* sums) {
  if constexpr (MODE == kC32 || MODE == kC32x) {
    float t[8];
#pragma unroll
    for (int v = 0; v < 8; ++v) t[v] = p[v] + p[v + 8];
#pragma unroll
    for (int v = 0; v < 4; ++v) t[v] += t[v + 4];
    sums[0] = pair_sum((t[0] + t[2]) + (t[1] + t[3]));
  } else if constexpr (MODE == kC16) {
    float s0 = p[0], s1 = p[8];
#pragma unroll
    for (int v = 1; v < 8; ++v) { s0 += p[v]; s1 += p[v + 8]; }
    sums[0] = pair_sum(s0);
    sums[1] = pair_sum(s1);
  } else if constexpr (MODE == kC8) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sums[i] = pair_sum((p[4 * i] + p[4 * i + 1]) + (p[4 * i + 2] + p[4 * i + 3]));
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

// Lane l of a wave holds logits of rows l%32 of both row tiles (mref[0..1]),
// and after pooling owns row l of the wave (row tile l/32): zsum and chunk_acc
// belong to that row.
struct RangeState {
  float mref[2];    // references of rows (tile 0, l%32) and (tile 1, l%32), scaled log2 units
  double zsum;      // own row: sum of the segment's chunk sums
  float chunk_acc;  // kC32x (c = 64, 96, ...): own row's running sum of the open chunk
  bool overflow;
};

// Sum over the lane pair (l, l^32) of one tile's value x0 (row tile 0) and
// x1 (row tile 1), delivered to the lane that owns the row: lanes 0..31 get
// x0[l] + x0[l+32], lanes 32..63 get x1[l-32] + x1[l].
__device__ __forceinline__ float own_row_sum(float x0, float x1) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_int(x0), __float_as_int(x1), false, false);
  return __int_as_float(r[0]) + __int_as_float(r[1]);
}

// kC4: chunk 2i+h of a subtile lives in lane half h.  After the swap lane l
// holds, for its own row, chunk 2i in lo and chunk 2i+1 in hi.
__device__ __forceinline__ void own_row_pair(float x0, float x1, float& lo, float& hi) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_int(x0), __float_as_int(x1), false, false);
  lo = __int_as_float(r[0]);
  hi = __int_as_float(r[1]);
}

// Pools the numerators p[rt] (keys past the segment end already zero) of one
// 32-key subtile starting at segment-relative key rk0 into per-chunk sums of the
// lane's own row, writes them to the partials and adds them to z.  Register v
// holds key 8*(v/4) + 4*half + v%4.  A short subtile writes zeros to chunk
// slots past the segment's last key; those slots exist (a row-block-head owns
// U*UK/c of them, UK a multiple of 64 and c) and nothing reads them.
template <int MODE>
__device__ __forceinline__ void pool_subtile(const ScoreArgs& a, const f32x16 (&p)[2], int rk0,
                                             int nkeys, float* part, int row, RangeState& st) {
  if constexpr (MODE == kC32 || MODE == kC32x) {
    float t[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      float u[8];
#pragma unroll
      for (int v = 0; v < 8; ++v) u[v] = p[rt][v] + p[rt][v + 8];
#pragma unroll
      for (int v = 0; v < 4; ++v) u[v] += u[v + 4];
      t[rt] = (u[0] + u[2]) + (u[1] + u[3]);
    }
    const float c = own_row_sum(t[0], t[1]);
    if constexpr (MODE == kC32) {
      part[(int64_t)(rk0 >> 5) * a.w.ldp + row] = c;
      st.zsum += (double)c;
    } else {
      st.chunk_acc += c;
      if ((rk0 + kSub) % a.c == 0 || rk0 + kSub >= nkeys) {  // uniform: the chunk closes
        part[(int64_t)(rk0 / a.c) * a.w.ldp + row] = st.chunk_acc;
        st.zsum += (double)st.chunk_acc;
        st.chunk_acc = 0.f;
      }
    }
  } else if constexpr (MODE == kC16) {
    // chunk 0: registers 0..7, chunk 1: registers 8..15
    float t[2][2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int b = 8 * h;
        t[rt][h] = ((p[rt][b] + p[rt][b + 1]) + (p[rt][b + 2] + p[rt][b + 3])) +
                   ((p[rt][b + 4] + p[rt][b + 5]) + (p[rt][b + 6] + p[rt][b + 7]));
      }
    const int jl0 = rk0 >> 4;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const float c = own_row_sum(t[0][h], t[1][h]);
      part[(int64_t)(jl0 + h) * a.w.ldp + row] = c;
      st.zsum += (double)c;
    }
  } else if constexpr (MODE == kC8) {
    // chunk i: registers 4i..4i+3
    const int jl0 = rk0 >> 3;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float t[2];
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
        t[rt] = (p[rt][4 * i] + p[rt][4 * i + 1]) + (p[rt][4 * i + 2] + p[rt][4 * i + 3]);
      const float c = own_row_sum(t[0], t[1]);
      part[(int64_t)(jl0 + i) * a.w.ldp + row] = c;
      st.zsum += (double)c;
    }
  } else {  // kC4: registers 4i..4i+3 of half h are chunk 2i+h
    const int jl0 = rk0 >> 2;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float t[2];
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
        t[rt] = (p[rt][4 * i] + p[rt][4 * i + 1]) + (p[rt][4 * i + 2] + p[rt][4 * i + 3]);
      float lo, hi;
      own_row_pair(t[0], t[1], lo, hi);
      part[(int64_t)(jl0 + 2 * i) * a.w.ldp + row] = lo;
      part[(int64_t)(jl0 + 2 * i + 1) * a.w.ldp + row] = hi;
      st.zsum += (double)lo;
      st.zsum += (double)hi;
    }
  }
}

// One 32-key subtile (segment-relative keys rk0 .. rk0+31 of a segment holding
// nkeys keys), read from LDS rows lrow0 .. lrow0+31.  FULL: all 32 keys valid
// (uniform; only a segment's last subtile can be short).  PASS 0 and PASS 2:
// partial sums against st.mref.  PASS 1: exact segment maximum only.
template <int D, int MODE, int PASS, bool FULL>
__device__ __forceinline__ void process_subtile(const ScoreArgs& a, const bf16x8 (&qf)[2][D / 16],
                                                const uint16_t* lds, int lrow0, int rk0, int nkeys,
                                                float* part, int my_row0, RangeState& st) {
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
      // references are whole numbers (log2 units): the fold rescales by exact
      // powers of two
      st.mref[rt] = fmaxf(st.mref[rt], ceilf(mx * a.c1));
    }
    return;
  }

  // p = exp2(c1*dot - mc); keys past the segment's end contribute 0
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
  pool_subtile<MODE>(a, acc, rk0, nkeys, part, my_row0 + lane, st);
}

// ---- software-pipelined steady state (PASS 0, full 64-key stages) ----------
// A stage is two subtiles.  Each subtile's 16 MFMAs are issued in the same
// scheduling region as the previous subtile's softmax VALU work (the compiler
// interleaves the two), and the last subtile's VALU work is carried over the
// stage barrier into the next stage.

// All 16 MFMAs of one subtile (both row tiles share each K fragment).  The
// fragment reads are left to the scheduler: reading all of them ahead costs
// 32 more VGPRs and measured slower.
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

// Softmax numerators of both row tiles of a full 32-key subtile starting at
// segment-relative key rk0, then pooling into the lane's own row.  Chunk sums
// are not checked here: all terms are >= 0, so z exceeds the guard (or is not
// finite) whenever one of its chunk sums does, and the segment is checked once
// at its end.
template <int MODE>
__device__ __forceinline__ void valu_subtile(const ScoreArgs& a, f32x16 (&acc)[2], int rk0,
                                             int nkeys, float* part, int row, RangeState& st) {
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    const float nm = -st.mref[rt];
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[rt][v] = __builtin_amdgcn_exp2f(fmaf(acc[rt][v], a.c1, nm));
  }
  pool_subtile<MODE>(a, acc, rk0, nkeys, part, row, st);
}

// One full 64-key stage as two slots.  Slot 0: MFMAs of subtile 0 with the
// VALU work of the subtile carried from the previous stage; slot 1: MFMAs of
// subtile 1 (into `carry`) with the VALU work of subtile 0.
template <int D, int MODE, bool CARRY>
__device__ __forceinline__ void fast_stage(const ScoreArgs& a, const bf16x8 (&qf)[2][D / 16],
                                           const uint16_t* cur, int rk0, int nkeys, float* part,
                                           int row, RangeState& st, f32x16 (&carry)[2],
                                           int& carry_rk) {
  f32x16 acc[2];
  __builtin_amdgcn_sched_barrier(0);
  mfma_subtile<D>(cur, 0, qf, acc);
  if constexpr (CARRY) {
    valu_subtile<MODE>(a, carry, carry_rk, nkeys, part, row, st);
  }
  __builtin_amdgcn_sched_barrier(0);
  mfma_subtile<D>(cur, kSub, qf, carry);
  valu_subtile<MODE>(a, acc, rk0, nkeys, part, row, st);
  __builtin_amdgcn_sched_barrier(0);
  carry_rk = rk0 + kSub;
}

// The first full stage of a segment: its first subtile's logits are already
// in `first` (the reference was taken from them), so only slot 1 remains --
// the second subtile's MFMAs beside the first subtile's VALU work.
template <int D, int MODE>
__device__ __forceinline__ void fast_stage_first(const ScoreArgs& a, const bf16x8 (&qf)[2][D / 16],
                                                 const uint16_t* cur, int rk0, int nkeys, float* part,
                                                 int row, RangeState& st, f32x16 (&first)[2],
                                                 f32x16 (&carry)[2], int& carry_rk) {
  __builtin_amdgcn_sched_barrier(0);
  mfma_subtile<D>(cur, kSub, qf, carry);
  valu_subtile<MODE>(a, first, rk0, nkeys, part, row, st);
  __builtin_amdgcn_sched_barrier(0);
  carry_rk = rk0 + kSub;
}

// Reference from a full subtile's logits: the scaled maximum of each row's,
// rounded up to a whole number.
__device__ __forceinline__ void reference_of(const ScoreArgs& a, const f32x16 (&acc)[2],
                                             RangeState& st) {
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    float mx = acc[rt][0];
#pragma unroll
    for (int v = 1; v < 16; ++v) mx = fmaxf(mx, acc[rt][v]);
    mx = fmaxf(mx, partner_f(mx));
    st.mref[rt] = ceilf(mx * a.c1);
  }
}

// Segment reference: the scaled maximum of each row's logits over the
// segment's first 32 keys (already in LDS buffer 0).
template <int D, int MODE>
__device__ __forceinline__ void segment_reference(const ScoreArgs& a, const bf16x8 (&qf)[2][D / 16],
                                                  const uint16_t* lds, int nkeys, int my_row0,
                                                  RangeState& st) {
  st.mref[0] = st.mref[1] = -INFINITY;
  process_subtile<D, MODE, 1, false>(a, qf, lds, 0, 0, nkeys, nullptr, my_row0, st);
}

template <int D>
__device__ __forceinline__ void load_q(const ScoreArgs& a, int g, int row0, bf16x8 (&qf)[2][D / 16]);

// PASS 0 over one segment (keys kbeg .. kbeg+nkeys-1 of KV head g): the
// reference from the first subtile, pipelined full stages, then the short tail
// stage (if any) through process_subtile.  Returns whether a chunk sum may have
// left the guard (then the fallback kernel redoes the segment exactly).
template <int D, int MODE>
__device__ __forceinline__ bool run_segment_fast(const ScoreArgs& a, int g, int64_t kbeg, int nkeys,
                                                 int row0, bf16x8 (&qf)[2][D / 16],
                                                 uint16_t* lds, RangeState& st) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nstage = (nkeys + kStage - 1) / kStage;
  const int nfull = nkeys / kStage;
  const int my_row0 = row0 + wave * kWaveRows;
  st.overflow = false;
  st.chunk_acc = 0.f;
  st.zsum = 0.0;
  float* part = a.part + ((int64_t)g * a.m_pad + kbeg / a.c) * a.w.ldp;

  const StageOffsets<D> o(a.Hkv, g);
  const int64_t stage_elems = (int64_t)kStage * a.Hkv * D;
  const uint16_t* kbase = a.k + kbeg * a.Hkv * D;
  constexpr int kBuf = kStage * SubtileLds<D>::kRow;  // elements per LDS stage buffer

  StageRegs<D> r;
  if (nfull > 0)
    stage_load_full<D>(kbase, o, r);
  else
    stage_load<D>(kbase, nkeys, o, r);
  // Q after the first stage's loads: loads return in order, so the stage's
  // LDS store and barrier do not wait for Q
  load_q<D>(a, g, row0, qf);
  if (nfull > 0)
    stage_store<D, true>(r, lds);
  else
    stage_store<D, false>(r, lds);
  __syncthreads();
  f32x16 carry[2], first[2];
  int carry_rk = 0;
  if (nfull > 0) {  // the first subtile's logits serve the reference and the first stage
    mfma_subtile<D>(lds, 0, qf, first);
    reference_of(a, first, st);
  } else {
    segment_reference<D, MODE>(a, qf, lds, nkeys, my_row0, st);
  }
  for (int s = 0; s < nfull; ++s) {
    const int rk0 = s * kStage;
    const uint16_t* next = kbase + (s + 1) * stage_elems;
    // uniform: the next stage is full, the short tail, or absent
    if (s + 1 < nfull)
      stage_load_full<D>(next, o, r);
    else if (s + 1 < nstage)
      stage_load<D>(next, nkeys - rk0 - kStage, o, r);
    const uint16_t* cur = lds + (s & 1) * kBuf;
    if (s == 0)
      fast_stage_first<D, MODE>(a, qf, cur, rk0, nkeys, part, my_row0 + lane, st, first, carry,
                                carry_rk);
    else
      fast_stage<D, MODE, true>(a, qf, cur, rk0, nkeys, part, my_row0 + lane, st, carry, carry_rk);
    uint16_t* nbuf = lds + ((s + 1) & 1) * kBuf;
    if (s + 1 < nfull)
      stage_store<D, true>(r, nbuf);
    else if (s + 1 < nstage)
      stage_store<D, false>(r, nbuf);
    __syncthreads();
  }
  if (nfull > 0) valu_subtile<MODE>(a, carry, carry_rk, nkeys, part, my_row0 + lane, st);
  if (nfull < nstage) {  // short last stage
    const int rk0 = nfull * kStage;
    const uint16_t* cur = lds + (nfull & 1) * kBuf;
    process_subtile<D, MODE, 0, false>(a, qf, cur, 0, rk0, nkeys, part, my_row0, st);
    if (rk0 + kSub < nkeys)
      process_subtile<D, MODE, 0, false>(a, qf, cur, kSub, rk0 + kSub, nkeys, part, my_row0, st);
  }
  st.overflow |= !(st.zsum <= (double)kOverflowGuard);
  return st.overflow;
}

// One plain pass over a segment (see process_subtile for PASS); used by the
// exact fallback kernel.
template <int D, int MODE, int PASS>
__device__ __forceinline__ void run_segment(const ScoreArgs& a, int g, int64_t kbeg, int nkeys,
                                            int row0, const bf16x8 (&qf)[2][D / 16], uint16_t* lds,
                                            RangeState& st) {
  const int wave = threadIdx.x >> 6;
  const int nstage = (nkeys + kStage - 1) / kStage;
  const int my_row0 = row0 + wave * kWaveRows;
  st.chunk_acc = 0.f;
  if (PASS != 1) st.zsum = 0.0;
  if (PASS == 1) st.mref[0] = st.mref[1] = -INFINITY;
  float* part = a.part + ((int64_t)g * a.m_pad + kbeg / a.c) * a.w.ldp;

  const StageOffsets<D> o(a.Hkv, g);
  const int64_t stage_elems = (int64_t)kStage * a.Hkv * D;
  const uint16_t* kbase = a.k + kbeg * a.Hkv * D;
  constexpr int kBuf = kStage * SubtileLds<D>::kRow;

  StageRegs<D> r;
  stage_load<D>(kbase, nkeys, o, r);
  stage_store<D, false>(r, lds);
  __syncthreads();
  for (int s = 0; s < nstage; ++s) {
    const int rk0 = s * kStage;
    if (s + 1 < nstage) stage_load<D>(kbase + (s + 1) * stage_elems, nkeys - rk0 - kStage, o, r);
    const uint16_t* cur = lds + (s & 1) * kBuf;
    if (rk0 + kStage <= nkeys) {
      process_subtile<D, MODE, PASS, true>(a, qf, cur, 0, rk0, nkeys, part, my_row0, st);
      process_subtile<D, MODE, PASS, true>(a, qf, cur, kSub, rk0 + kSub, nkeys, part, my_row0, st);
    } else {
      process_subtile<D, MODE, PASS, false>(a, qf, cur, 0, rk0, nkeys, part, my_row0, st);
      if (rk0 + kSub < nkeys)
        process_subtile<D, MODE, PASS, false>(a, qf, cur, kSub, rk0 + kSub, nkeys, part, my_row0, st);
    }
    if (s + 1 < nstage) stage_store<D, false>(r, lds + ((s + 1) & 1) * kBuf);
    __syncthreads();
  }
}

// Q^T fragments of a row block: B operand, lane l holds row l%32 of a row tile
// and d = 16*ks + 8*half .. +7 (zero past R).
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

// Reference and sum of every row of the block for segment slot s of rbh (rows
// past R hold zero queries and are written too: the arrays span whole blocks).
__device__ __forceinline__ void store_stats(const ScoreArgs& a, int rbh, int s, const RangeState& st) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // both lane halves hold both references: the swap hands lane l its own row's
  float ref, unused;
  own_row_pair(st.mref[0], st.mref[1], ref, unused);
  const int64_t o = ((int64_t)rbh * a.w.NS + s) * kBlockRows + wave * kWaveRows + lane;
  a.mc[o] = ref;
  a.z[o] = st.zsum;
}

// Segment s of row block rbh: keys kbeg .. kbeg+nkeys-1.
struct Segment {
  int rbh, s;
  int64_t kbeg;
  int nkeys;
};
__device__ __forceinline__ Segment segment_at(const ScoreWork& wk, int64_t n, int rbh, int s) {
  Segment g;
  g.rbh = rbh;
  g.s = s;
  g.kbeg = (int64_t)wk.seg_begin(s) * wk.UK;
  g.nkeys = (int)(min<int64_t>((int64_t)wk.seg_begin(s + 1) * wk.UK, n) - g.kbeg);
  return g;
}

// Workgroup w (logical) runs row block rb of KV head g at segment s, with rb
// varying fastest: the workgroups that read the same keys are adjacent, hence
// on the same XCD and its L2.
__device__ __forceinline__ Segment segment_of(const ScoreWork& wk, int64_t n, int w) {
  const int rb = w % wk.RB, s = (w / wk.RB) % wk.NS, g = w / (wk.RB * wk.NS);
  return segment_at(wk, n, g * wk.RB + rb, s);
}

// Fold of the segments of row block rbh: thread t owns row t of the block
// (rows past R fold too; nothing reads them).  M = max mc, Z = sum
// exp2(mc - M) z, and each segment's z slot becomes its weight exp2(mc - M)/Z.
// Up to kFoldBatch segments are held in registers, loaded in one round trip;
// more are read in batches of kFoldBatch (three passes).
constexpr int kFoldBatch = 32;

// exp2(mc - M) for whole-number references mc <= M: an exact power of two
// (zero once it is below the smallest subnormal).
__device__ __forceinline__ double seg_factor(float mc, float M) {
  return mc == M ? 1.0 : ldexp(1.0, (int)fmaxf(mc - M, -1100.f));
}

struct FoldRegs {
  float v[kFoldBatch];
  double zz[kFoldBatch];
};

// This thread's row of every segment (NS <= kFoldBatch); absent segments read
// as (-inf, 0), which contribute exactly 0.
__device__ __forceinline__ void fold_load(const float* mc, const double* z, const ScoreWork& wk,
                                          int rbh, FoldRegs& r) {
  const int64_t base = (int64_t)rbh * wk.NS * wk.rpb + threadIdx.x;
#pragma unroll
  for (int i = 0; i < kFoldBatch; ++i) {
    const bool ok = i < wk.NS;
    r.v[i] = ok ? mc[base + (int64_t)i * wk.rpb] : -INFINITY;
    r.zz[i] = ok ? z[base + (int64_t)i * wk.rpb] : 0.0;
  }
}

__device__ __forceinline__ void fold_apply(double* z, const ScoreWork& wk, int rbh,
                                           const FoldRegs& r) {
  const int64_t base = (int64_t)rbh * wk.NS * wk.rpb + threadIdx.x;
  float M = -INFINITY;
#pragma unroll
  for (int i = 0; i < kFoldBatch; ++i) M = fmaxf(M, r.v[i]);
  double Z = 0.0;  // ascending segment order
#pragma unroll
  for (int i = 0; i < kFoldBatch; ++i) Z += seg_factor(r.v[i], M) * r.zz[i];
  const double inv = 1.0 / Z;
#pragma unroll
  for (int i = 0; i < kFoldBatch; ++i)
    if (i < wk.NS) z[base + (int64_t)i * wk.rpb] = seg_factor(r.v[i], M) * inv;
}

// More than kFoldBatch segments: the same sums, in the same order, in batches.
__device__ __forceinline__ void fold_row_block_batched(const float* mc, double* z,
                                                       const ScoreWork& wk, int rbh) {
  const int64_t base = (int64_t)rbh * wk.NS * wk.rpb + threadIdx.x;
  const int NS = wk.NS, rpb = wk.rpb;
  float M = -INFINITY;
  for (int s0 = 0; s0 < NS; s0 += kFoldBatch) {
    float v[kFoldBatch];
#pragma unroll
    for (int i = 0; i < kFoldBatch; ++i)
      v[i] = s0 + i < NS ? mc[base + (int64_t)(s0 + i) * rpb] : -INFINITY;
#pragma unroll
    for (int i = 0; i < kFoldBatch; ++i) M = fmaxf(M, v[i]);
  }
  double Z = 0.0;
  for (int s0 = 0; s0 < NS; s0 += kFoldBatch) {
    float v[kFoldBatch];
    double zz[kFoldBatch];
#pragma unroll
    for (int i = 0; i < kFoldBatch; ++i) {
      const bool ok = s0 + i < NS;
      v[i] = ok ? mc[base + (int64_t)(s0 + i) * rpb] : -INFINITY;
      zz[i] = ok ? z[base + (int64_t)(s0 + i) * rpb] : 0.0;
    }
#pragma unroll
    for (int i = 0; i < kFoldBatch; ++i) Z += seg_factor(v[i], M) * zz[i];
  }
  const double inv = 1.0 / Z;
  for (int s0 = 0; s0 < NS; s0 += kFoldBatch) {
    float v[kFoldBatch];
#pragma unroll
    for (int i = 0; i < kFoldBatch; ++i) v[i] = s0 + i < NS ? mc[base + (int64_t)(s0 + i) * rpb] : M;
#pragma unroll
    for (int i = 0; i < kFoldBatch; ++i)
      if (s0 + i < NS) z[base + (int64_t)(s0 + i) * rpb] = seg_factor(v[i], M) * inv;
  }
}

__device__ __forceinline__ void fold_row_block(const float* mc, double* z, const ScoreWork& wk,
                                               int rbh) {
  if (wk.NS <= kFoldBatch) {
    FoldRegs r;
    fold_load(mc, z, wk, rbh, r);
    fold_apply(z, wk, rbh, r);
  } else {
    fold_row_block_batched(mc, z, wk, rbh);
  }
}

// Main pass: every workgroup runs its segment, pipelined, against the
// segment's own reference, and records whether a chunk sum left the guard.
template <int D, int MODE>
__global__ __launch_bounds__(kWaves * 64, 2) void score_bf16_kernel(ScoreArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * kStage * SubtileLds<D>::kRow];
  const uint32_t w = xcd_remap(blockIdx.x, a.nwg_padded);
  if (w >= a.nwg) return;
  // timing mode: each workgroup's start and end from the 100 MHz realtime
  // counter, one 16-byte store per workgroup
  const unsigned long long t_start = a.tstamp ? __builtin_amdgcn_s_memrealtime() : 0;
  const Segment sg = segment_of(a.w, a.n, (int)w);
  const int g = sg.rbh / a.w.RB, row0 = (sg.rbh % a.w.RB) * kBlockRows;
  bf16x8 qf[2][D / 16];  // loaded by run_segment_fast
  RangeState st;
  const bool of = run_segment_fast<D, MODE>(a, g, sg.kbeg, sg.nkeys, row0, qf, lds, st);
  const int any_of = __syncthreads_or(of ? 1 : 0);
  if (threadIdx.x == 0) a.flags[sg.rbh * a.w.NS + sg.s] = any_of;
  store_stats(a, sg.rbh, sg.s, st);
  if (a.tstamp) {
    __syncthreads();
    if (threadIdx.x == 0) {
      const unsigned long long t_end = __builtin_amdgcn_s_memrealtime();
      *reinterpret_cast<ulonglong2*>(a.tstamp + 2 * w) = make_ulonglong2(t_start, t_end);
    }
  }
}

// Fold pass, one workgroup per row block: redoes exactly (against its own
// maximum, two passes) any of the block's segments whose chunk sums left the
// guard in the main pass -- almost never -- then folds the block's segments.
template <int D, int MODE>
__global__ __launch_bounds__(kWaves * 64) void score_fold_kernel(ScoreArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * kStage * SubtileLds<D>::kRow];
  const int rbh = blockIdx.x;
  const int g = rbh / a.w.RB, row0 = (rbh % a.w.RB) * kBlockRows;
  // all flags of the block, and (speculatively) the block's statistics, in one
  // round trip; nothing flagged is the common case
  const bool in_regs = a.w.NS <= kFoldBatch;
  FoldRegs r;
  if (in_regs) fold_load(a.mc, a.z, a.w, rbh, r);
  int any = 0;
  for (int s = threadIdx.x; s < a.w.NS; s += blockDim.x) any |= a.flags[rbh * a.w.NS + s];
  const bool redo = __syncthreads_or(any);
  if (redo) {
    for (int s = 0; s < a.w.NS; ++s) {
      if (!a.flags[rbh * a.w.NS + s]) continue;  // uniform
      const Segment o = segment_at(a.w, a.n, rbh, s);
      bf16x8 qf[2][D / 16];
      load_q<D>(a, g, row0, qf);
      RangeState st;
      run_segment<D, MODE, 1>(a, g, o.kbeg, o.nkeys, row0, qf, lds, st);
      run_segment<D, MODE, 2>(a, g, o.kbeg, o.nkeys, row0, qf, lds, st);
      store_stats(a, rbh, s, st);
      __syncthreads();
    }
  }
  if (!in_regs) {
    fold_row_block_batched(a.mc, a.z, a.w, rbh);
    return;
  }
  if (redo) fold_load(a.mc, a.z, a.w, rbh, r);  // this thread's rows, as redone
  fold_apply(a.z, a.w, rbh, r);
}

// fp32 path: the main kernel already redid overflowing segments; fold only.
__global__ __launch_bounds__(kWaveRows) void score_fold_f32_kernel(const float* __restrict__ mc,
                                                                   double* __restrict__ z,
                                                                   ScoreWork wk) {
  fold_row_block(mc, z, wk, blockIdx.x);
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
  int64_t n, m_pad;
  int S, Hq, Hkv, G, R, c;
  float c1;
  ScoreWork w;
  int nwg;
};

template <int D, int MODE, int PASS>
__device__ bool run_span_f32(const ScoreArgsF32& a, int g, int64_t kbeg, int64_t kend, int row0,
                             const float (&qf)[2][D / 2], float (&mref)[2], double (&zsum)[2]) {
  const int lane = threadIdx.x & 63, half = lane >> 5;
  const int nsub = (int)((kend - kbeg + kSub - 1) / kSub);
  bool overflow = false;
  float chunk_acc[2] = {0.f, 0.f};
  if (PASS != 1) { zsum[0] = 0.0; zsum[1] = 0.0; }
  if (PASS == 1) { mref[0] = -INFINITY; mref[1] = -INFINITY; }
  float* part = a.part + ((int64_t)g * a.m_pad + kbeg / a.c) * a.w.ldp;
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
          mref[rt] = fmaxf(mref[rt], ceilf(mx * a.c1));
        else
          mref[rt] = ceilf(mx * a.c1);
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
        if (row < a.R) part[(int64_t)jl * a.w.ldp + row] = mine;
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
            if (row < a.R && key_first < nvalid) part[(int64_t)jl * a.w.ldp + row] = sums[i];
          }
        } else if (rt == half) {
          const int row = row0 + rt * 32 + (lane & 31);
#pragma unroll
          for (int i = 0; i < kN; ++i) {
            int key_first = i * (kSub / kN);
            if (row < a.R && key_first < nvalid) part[(int64_t)(jl0 + i) * a.w.ldp + row] = sums[i];
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
  const int w = blockIdx.x;
  if (w >= a.nwg) return;
  const int lane = threadIdx.x & 63, half = lane >> 5;
  const Segment sg = segment_of(a.w, a.n, w);
  const int g = sg.rbh / a.w.RB, row0 = (sg.rbh % a.w.RB) * kWaveRows;
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
  const int64_t kend = sg.kbeg + sg.nkeys;
  bool of = run_span_f32<D, MODE, 0>(a, g, sg.kbeg, kend, row0, qf, mref, zsum);
  // one wave: the decision is wave-uniform via a ballot
  if (__any(of)) {
    run_span_f32<D, MODE, 1>(a, g, sg.kbeg, kend, row0, qf, mref, zsum);
    run_span_f32<D, MODE, 2>(a, g, sg.kbeg, kend, row0, qf, mref, zsum);
  }
  const int64_t o = ((int64_t)sg.rbh * a.w.NS + sg.s) * kWaveRows + lane;
  a.mc[o] = half ? mref[1] : mref[0];
  a.z[o] = half ? zsum[1] : zsum[0];
}

// ---------------------------------------------------------------------------
// finalize
// ---------------------------------------------------------------------------
// Reduction: A_j = sum over KV heads g (in order) of sum over rows r of
// w[segment holding chunk j][r] * P[g][j][r], in fp64.  One workgroup of 256
// threads per chunk: thread i takes rows 4i .. 4i+3, 4i+1024 .. of every head
// in order (16-byte partial loads, 32-byte weight loads), then a fixed tree
// over LDS reduces the 256 sums.
constexpr int kReduceThreads = 256;
constexpr int kReduceWide = 4;       // chunks per workgroup of the many-chunk reduction
constexpr int kReduceUnroll = 4;     // (head, row group) pairs per step
constexpr int64_t kReduceWideChunks = 4096;  // chunk count from which it is used

__global__ __launch_bounds__(kReduceThreads) void chunk_reduce_kernel(
    const float* __restrict__ part, const double* __restrict__ w, double* __restrict__ A,
    ScoreWork wk, int Hkv, int R, int64_t m_pad, int c, int log2_rpb) {
  __shared__ double red[kReduceThreads];
  const int64_t j = blockIdx.x;
  const int tid = threadIdx.x;
  const int seg = wk.seg_of_unit((int)(j * c / wk.UK));  // the same for every row block
  double s = 0.0;
#pragma unroll 2
  for (int g = 0; g < Hkv; ++g) {
    const float* p = part + ((int64_t)g * m_pad + j) * wk.ldp;
    for (int r = 4 * tid; r < R; r += 4 * kReduceThreads) {
      // ldp and rpb are multiples of 64: the 4 rows are in bounds and in one block
      const f32x4 pv = *reinterpret_cast<const f32x4*>(p + r);
      const int rbh = g * wk.RB + (r >> log2_rpb);
      const double* wr = w + ((int64_t)rbh * wk.NS + seg) * wk.rpb + (r & (wk.rpb - 1));
      const double2 w01 = *reinterpret_cast<const double2*>(wr);
      const double2 w23 = *reinterpret_cast<const double2*>(wr + 2);
      if (r + 3 < R) {
        s += (double)pv[0] * w01.x;
        s += (double)pv[1] * w01.y;
        s += (double)pv[2] * w23.x;
        s += (double)pv[3] * w23.y;
      } else {
        const double wv[4] = {w01.x, w01.y, w23.x, w23.y};
        for (int e = 0; e < 4 && r + e < R; ++e) s += (double)pv[e] * wv[e];
      }
    }
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

// The same reduction for many chunks: NJ consecutive chunks per workgroup,
// which share each weight load while they lie in one segment (SAME), and a
// flat walk over (head, 4-row group) pairs, UNR pairs per step with all their
// loads issued before any is used (indices clamped, so no load waits on a
// predicate).  Each chunk's sum takes its terms in a fixed order (thread i:
// pairs i, i + 256, ...), then a fixed tree over LDS.
template <int NJ, int UNR, bool SAME>
__device__ __forceinline__ void reduce_flat_sums(const float* __restrict__ part,
                                                 const double* __restrict__ w, const ScoreWork& wk,
                                                 int Hkv, int R, int64_t m_pad, int log2_rpb,
                                                 const int64_t (&jc)[NJ], const int (&seg)[NJ],
                                                 double (&s)[NJ]) {
  constexpr int NW = SAME ? 1 : NJ;  // weight sets per pair
  const int nq = (R + 3) / 4;        // 4-row groups per head
  const int total = Hkv * nq;
  for (int base = threadIdx.x; base < total; base += UNR * kReduceThreads) {
    f32x4 pv[UNR][NJ];
    double wv[UNR][NW][4];
    int rr[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int idx = min(base + u * kReduceThreads, total - 1);
      const int g = idx / nq, r = 4 * (idx - g * nq);
      rr[u] = r;
      const float* p = part + (int64_t)g * m_pad * wk.ldp + r;
#pragma unroll
      for (int q = 0; q < NJ; ++q) pv[u][q] = *reinterpret_cast<const f32x4*>(p + jc[q] * wk.ldp);
      const int rbh = g * wk.RB + (r >> log2_rpb);
      const double* wb = w + (int64_t)rbh * wk.NS * wk.rpb + (r & (wk.rpb - 1));
#pragma unroll
      for (int q = 0; q < NW; ++q) {
        const double* wr = wb + (int64_t)seg[q] * wk.rpb;
        const double2 w01 = *reinterpret_cast<const double2*>(wr);
        const double2 w23 = *reinterpret_cast<const double2*>(wr + 2);
        wv[u][q][0] = w01.x; wv[u][q][1] = w01.y; wv[u][q][2] = w23.x; wv[u][q][3] = w23.y;
      }
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      if (base + u * kReduceThreads >= total) break;
      const int r = rr[u];
#pragma unroll
      for (int q = 0; q < NJ; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (r + e < R) s[q] += (double)pv[u][q][e] * wv[u][SAME ? 0 : q][e];
    }
  }
}

template <int NJ, int UNR>
__global__ __launch_bounds__(kReduceThreads) void chunk_reduce_flat_kernel(
    const float* __restrict__ part, const double* __restrict__ w, double* __restrict__ A,
    ScoreWork wk, int Hkv, int R, int64_t m, int64_t m_pad, int c, int log2_rpb) {
  __shared__ double red[NJ][kReduceThreads];
  const int64_t j0 = (int64_t)blockIdx.x * NJ;
  const int tid = threadIdx.x;
  int64_t jc[NJ];
  int seg[NJ];
  bool same = true;
#pragma unroll
  for (int q = 0; q < NJ; ++q) {
    jc[q] = j0 + q < m ? j0 + q : m - 1;
    seg[q] = wk.seg_of_unit((int)(jc[q] * c / wk.UK));
    same = same && seg[q] == seg[0];
  }
  double s[NJ];
#pragma unroll
  for (int q = 0; q < NJ; ++q) s[q] = 0.0;
  if (same)  // uniform
    reduce_flat_sums<NJ, UNR, true>(part, w, wk, Hkv, R, m_pad, log2_rpb, jc, seg, s);
  else  // a workgroup across a segment boundary: one pair per step (the order is the same)
    reduce_flat_sums<NJ, 1, false>(part, w, wk, Hkv, R, m_pad, log2_rpb, jc, seg, s);
#pragma unroll
  for (int q = 0; q < NJ; ++q) red[q][tid] = s[q];
  __syncthreads();
#pragma unroll
  for (int width = kReduceThreads / 2; width >= 64; width >>= 1) {
    if (tid < width) {
#pragma unroll
      for (int q = 0; q < NJ; ++q) red[q][tid] += red[q][tid + width];
    }
    __syncthreads();
  }
  if (tid < 64) {
#pragma unroll
    for (int q = 0; q < NJ; ++q) {
      double x = red[q][tid];
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
      if (tid == 0 && j0 + q < m) A[j0 + q] = x;
    }
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
  const bool f32 = d->dtype == CKV_DTYPE_F32;
  const int64_t c = d->chunk_size;
  p.m = ceil_div(d->n_prefix, c);
  p.rows = G * d->n_suffix;
  ScoreWork& w = p.w;
  w.rpb = f32 ? kWaveRows : kBlockRows;
  w.RB = (int32_t)ceil_div(p.rows, w.rpb);
  int64_t g64 = 64, cc = c;  // gcd(64, c)
  while (cc) { const int64_t t = g64 % cc; g64 = cc; cc = t; }
  const int64_t UK = 64 / g64 * c;  // lcm(64, c)
  const int64_t U = ceil_div(d->n_prefix, UK);
  const int64_t H_RB = (int64_t)d->n_kv_heads * w.RB;
  // A fixed grid target (two 256-thread workgroups per CU of a 256-CU MI355X
  // for bf16) keeps the decomposition, and so every rounding, independent of
  // the device the library runs on.  Segments of the pipelined bf16 kernel
  // keep at least 4 stages while the fold still holds a row's segments in
  // registers (kFoldBatch), else at least 8; the one-wave fp32 kernel's keep
  // 64 keys.
  const int64_t target = f32 ? 1024 : 512;
  const int64_t NS_max = std::max<int64_t>(1, target / H_RB);
  auto segments = [&](int64_t min_keys) {
    const int64_t min_units = std::max<int64_t>(1, min_keys / UK);
    return std::min<int64_t>(NS_max, std::max<int64_t>(1, U / min_units));
  };
  int64_t NS = segments(f32 ? 64 : 256);
  if (!f32 && NS > kFoldBatch) NS = segments(512);
  // bytes == 0 marks an unsupported shape
  if (UK > INT32_MAX || U > INT32_MAX || H_RB * NS >= (int64_t(1) << 31)) return p;
  w.UK = (int32_t)UK;
  w.U = (int32_t)U;
  w.NS = (int32_t)NS;
  w.ldp = w.RB * w.rpb;
  const size_t H = (size_t)d->n_kv_heads, m_pad = (size_t)(U * UK / c);
  const size_t stats = (size_t)H_RB * NS * (size_t)w.rpb;
  size_t off = 0;
  p.off_part = off;
  off = align_up(off + H * m_pad * (size_t)w.ldp * sizeof(float), 256);
  p.off_mc = off;
  off = align_up(off + stats * sizeof(float), 256);
  p.off_z = off;
  off = align_up(off + stats * sizeof(double), 256);
  p.off_flags = off;
  off = align_up(off + (size_t)H_RB * NS * sizeof(int), 256);
  p.bytes = off;
  return p;
}

int64_t score_span_words(const ckv_dims* d) {
  const ScorePlan p = make_score_plan(d);
  return 2 * (int64_t)d->n_kv_heads * p.w.RB * p.w.NS;
}

ckv_status launch_score(const ckv_dims* d, const void* q, const void* k, double* scores, void* ws,
                        size_t ws_bytes, hipStream_t st, hipEvent_t main_stop,
                        unsigned long long* main_span) {
  const ScorePlan p = make_score_plan(d);
  if (p.bytes == 0) CKV_FAIL(CKV_EUNSUPPORTED, "shape too large for the scoring decomposition");
  if (ws_bytes < p.bytes) CKV_FAIL(CKV_EINVAL, "score workspace too small: %zu < %zu", ws_bytes, p.bytes);
  const int mode = chunk_mode(d->chunk_size);
  char* base = static_cast<char*>(ws);
  float* part = reinterpret_cast<float*>(base + p.off_part);
  float* mc = reinterpret_cast<float*>(base + p.off_mc);
  double* z = reinterpret_cast<double*>(base + p.off_z);
  const int G = d->n_q_heads / d->n_kv_heads;
  const float c1 = resolve_scale(d) * 1.4426950408889634f;
  const int64_t m_pad = (int64_t)p.w.U * p.w.UK / d->chunk_size;
  const uint32_t nwg = (uint32_t)((int64_t)d->n_kv_heads * p.w.RB * p.w.NS);

  if (d->dtype == CKV_DTYPE_BF16) {
    ScoreArgs a;
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.part = part; a.mc = mc; a.z = z;
    a.flags = reinterpret_cast<int*>(base + p.off_flags);
    a.n = d->n_prefix; a.m_pad = m_pad;
    a.S = d->n_suffix; a.Hq = d->n_q_heads; a.Hkv = d->n_kv_heads; a.G = G;
    a.R = p.rows; a.c = d->chunk_size; a.c1 = c1; a.w = p.w;
    a.nwg = nwg;
    a.nwg_padded = (uint32_t)align_up(nwg, 8);
    a.tstamp = main_span;
    dim3 grid(a.nwg_padded), block(kWaves * 64);
    const dim3 fold_grid((unsigned)(d->n_kv_heads * p.w.RB));
#define CKV_SCORE_LAUNCH(DD, MM)                                                           \
  do {                                                                                     \
    hipLaunchKernelGGL((score_bf16_kernel<DD, MM>), grid, block, 0, st, a);                \
    if (main_stop) CKV_HIP(hipEventRecord(main_stop, st));                                \
    hipLaunchKernelGGL((score_fold_kernel<DD, MM>), fold_grid, block, 0, st, a);           \
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
    a.n = d->n_prefix; a.m_pad = m_pad;
    a.S = d->n_suffix; a.Hq = d->n_q_heads; a.Hkv = d->n_kv_heads; a.G = G;
    a.R = p.rows; a.c = d->chunk_size; a.c1 = c1; a.w = p.w;
    a.nwg = (int)nwg;
    dim3 grid(nwg), block(64);
    switch (mode) {
      case kC4: hipLaunchKernelGGL((score_f32_kernel<64, kC4>), grid, block, 0, st, a); break;
      case kC8: hipLaunchKernelGGL((score_f32_kernel<64, kC8>), grid, block, 0, st, a); break;
      case kC16: hipLaunchKernelGGL((score_f32_kernel<64, kC16>), grid, block, 0, st, a); break;
      case kC32: hipLaunchKernelGGL((score_f32_kernel<64, kC32>), grid, block, 0, st, a); break;
      default: hipLaunchKernelGGL((score_f32_kernel<64, kC32x>), grid, block, 0, st, a); break;
    }
    if (main_span) CKV_FAIL(CKV_EUNSUPPORTED, "in-kernel timing is for the bf16 path");
    if (main_stop) CKV_HIP(hipEventRecord(main_stop, st));
    hipLaunchKernelGGL(score_fold_f32_kernel, dim3((unsigned)(d->n_kv_heads * p.w.RB)),
                       dim3(kWaveRows), 0, st, mc, z, p.w);
  }
  CKV_HIP(hipGetLastError());
  const int log2_rpb = p.w.rpb == 256 ? 8 : 6;
  // one chunk per workgroup while the chunks are few (the reduction is bound
  // by load latency); with many chunks (the partials then run to hundreds of
  // MB) kReduceWide chunks per workgroup share each weight load
  if (p.m < kReduceWideChunks)
    hipLaunchKernelGGL(chunk_reduce_kernel, dim3((unsigned)p.m), dim3(kReduceThreads), 0, st, part,
                       z, scores, p.w, d->n_kv_heads, p.rows, m_pad, d->chunk_size, log2_rpb);
  else
    hipLaunchKernelGGL((chunk_reduce_flat_kernel<kReduceWide, kReduceUnroll>),
                       dim3((unsigned)ceil_div(p.m, kReduceWide)), dim3(kReduceThreads), 0, st,
                       part, z, scores, p.w, d->n_kv_heads, p.rows, p.m, m_pad, d->chunk_size,
                       log2_rpb);
  CKV_HIP(hipGetLastError());
  return CKV_OK;
}

}  // namespace ckv
