// attn.hip -- Re-Prefill sparse attention (Def. 2.1) for gfx950, bf16.
//
// For query t of head h (KV head g = h / G) the keys are the tokens of the k
// kept chunks (compact positions 0 .. k*c-1; rows past n of a short last chunk
// are masked) followed by the suffix tokens 0..t (causal).
//
// Rows of one KV head are r = t*G + i (query t, head g*G + i), so the G query
// heads that share a KV head share every K/V tile.  A workgroup owns 128 rows
// (4 waves x 32) and one contiguous slice ("split") of the key positions.  At
// its start it resolves every key of its slice to a source code (a prefix row
// of the K/V source, a suffix token, or no key) in LDS, so the tile loads are
// branch-free.  Per 64-key stage:
//   S^T = K Q^T   bf16 MFMA 32x32x16, A = K rows from LDS, B = Q^T in
//                 registers: every lane owns one query row and 16 keys;
//   online softmax in fp32 (exp2 with sm_scale*log2 e folded in) with a lazy
//                 reference: it moves only when a stage's maximum exceeds it
//                 by more than 2^8, so most stages skip the O rescale;
//   O^T += V^T P^T  A = V^T read from LDS with the transposing
//                 ds_read_b64_tr_b16, B = P^T straight from the softmax
//                 registers.
// The K operand rows are loaded in a permuted order so that the registers a
// lane holds after the first product are exactly the 8 consecutive keys the
// second product needs from it -- no register shuffles between the two.
// Splits write their normalised partial output O/l in bf16 (the output's own
// type and range) plus (reference, l) in fp32; a combine kernel merges them in
// split order (deterministic).

#include <atomic>

#include "ckv_internal.h"

namespace ckv {
namespace {

std::atomic<int> g_force_wide{0};  // ckv_debug_attn_wide_addressing

constexpr int kWaves = 4;
constexpr int kWaveRows = 32;
constexpr int kBlockRows = kWaves * kWaveRows;  // 128
constexpr int kTile = 64;                       // keys per LDS stage
constexpr int kSub = 32;                        // keys per MFMA product
constexpr int kMaxSliceKeys = 1024;             // keys per workgroup slice (8 KiB of key tables)
constexpr float kLazy = 8.f;                    // headroom of the lazy softmax reference (log2 units)
// Key tables: for every key of a slice, the row of its K/V source (as a byte
// offset from the source's base when all of them fit in 32 bits) and its
// visibility threshold -- a query t sees the key iff t >= thr.  thr = -1 marks
// a row of the prefix source (seen by every query); a suffix token p has
// thr = p (causal) and a row of the suffix source; a padding key has
// thr = kNever and suffix row 0 (always present; its weight is forced to 0).
constexpr int kPrefix = -1;
constexpr int kNever = 0x7fffffff;

// MFMA row p of the K operand holds key kappa(p); afterwards register v of a
// lane in half h holds key 16*(v/8) + 8*h + v%8.
__device__ __forceinline__ int kappa(int p) {
  const int i = p >> 3, h = (p >> 2) & 1, j = p & 3;
  return 16 * (i >> 1) + 8 * h + 4 * (i & 1) + j;
}

// K stage: rows padded by one 16-byte segment, so the operand reads (16
// consecutive lanes = 16 distinct rows, same segment) start 4 banks apart and
// every fragment is an immediate offset from one per-lane base.
template <int D>
struct KLds {
  static constexpr int kRow = D + 8;
};

// V stage: XOR swizzle of 16-byte segments, conflict-free for the transposing
// reads.
template <int D>
__device__ __forceinline__ int v_swz(int row) {
  if constexpr (D == 128)
    return ((row & 1) ? 4 : 0) ^ ((row & 2) ? 10 : 0);
  else
    return ((row & 1) ? 2 : 0) ^ ((row & 2) ? 4 : 0);
}
template <int D>
__device__ __forceinline__ int v_off(int row, int seg) { return row * D + ((seg ^ v_swz<D>(row)) << 3); }

__device__ __forceinline__ float partner_f(float x) {
  int v = __float_as_int(x);
  auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return __int_as_float(threadIdx.x & 32 ? r[0] : r[1]);
}

struct AttnArgs {
  const uint16_t* q;       // [S][Hq][D]
  const uint16_t* kbase;   // prefix chunks (see ChunkSource)
  const uint16_t* vbase;
  const int32_t* chunk_off;
  int32_t direct;
  int rows_per_slot;       // chunk slot stride of the source in rows of Hkv*D elements
  const int32_t* sel;      // [k]
  int kc;                  // k * c prefix positions (< 2^31)
  int64_t n, m;
  int c;
  int log2c;               // log2(c) when c is a power of two, else -1
  const uint16_t* ks;      // [S][Hkv][D]
  const uint16_t* vs;
  uint16_t* out;           // [S][Hq][D]
  uint16_t* o_part;        // [splits][Hkv][R][D]: O / l, bf16
  float2* ml_part;         // [splits][Hkv][R]: (reference, sum)
  int S, Hq, Hkv, G, R, n_splits, tiles_per_split, n_row_blocks;
  int partial;             // write split partials for a combine (else the output itself)
  int with_suffix;         // the keys end with the causal suffix (else prefix chunks only)
  float c1;
  uint32_t nblocks, nblocks_padded;
  uint32_t row_bytes;      // Hkv * D * 2: bytes between consecutive rows of a source
  int off32;               // every row of both sources lies below 4 GiB from its base
  uint32_t pre_bytes, suf_bytes;  // bytes of the prefix and suffix sources (when off32)
};

// Buffer resource over `bytes` bytes from p (raw loads; offsets past the end read 0).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// Table entries of compact key position pos, in two steps so that a workgroup
// can issue all its index loads before using any: key_chunk_loads fetches
// sel[u] (and the slot table entry) of the key's chunk u, key_entry finishes.
// Row off of kept chunk u sits at source row slot*rows_per_slot + off, slot =
// chunk_off[u] (slot table), sel[u] (spans read in place) or u (compact
// copy).
__device__ __forceinline__ int chunk_of(const AttnArgs& a, int pos) {
  return a.log2c >= 0 ? (pos >> a.log2c) : (int)((uint32_t)pos / (uint32_t)a.c);
}

__device__ __forceinline__ void key_chunk_loads(const AttnArgs& a, int pos, int& j, int& slot) {
  j = 0;
  slot = 0;
  if (pos < a.kc) {
    const int u = chunk_of(a, pos);
    j = a.sel[u];
    if (a.chunk_off) slot = a.chunk_off[u];
  }
}

__device__ __forceinline__ void key_entry(const AttnArgs& a, int pos, int j, int slot_tab, int& row,
                                          int& thr) {
  row = 0;
  thr = kNever;
  if (pos < a.kc) {
    const int u = chunk_of(a, pos);
    const int off = pos - u * a.c;
    if (j < 0 || (int64_t)j >= a.m) return;
    if ((int64_t)j * a.c + off >= a.n) return;  // past n in a short last chunk
    const int slot = a.chunk_off ? slot_tab : (a.direct ? j : u);
    row = slot * a.rows_per_slot + off;
    thr = kPrefix;
  } else if (pos < a.kc + a.S) {
    row = pos - a.kc;
    thr = row;
  }
}

// The K/V rows of one 64-key stage, fetched into registers (while the previous
// stage is consumed from LDS) and then written to the other LDS buffer.  Each
// thread moves kPer 16-byte pieces of K and of V: piece p is segment tid %
// kSegs of key tid / kSegs + p * kKeyStep.
template <int D>
struct TileRegs {
  static constexpr int kSegs = D / 8;
  static constexpr int kPer = kTile * kSegs / (kWaves * 64);  // 16-byte pieces per thread
  static constexpr int kKeyStep = kWaves * 64 / kSegs;
  u32x4 k[kPer], v[kPer];
};

// The table entries of this thread's keys of one stage (read one stage ahead,
// so the row loads never wait on LDS): the row's byte offset from its source's
// base (AttnArgs::off32) or the row itself, and the threshold.
template <int D>
struct TileKeys {
  int row[TileRegs<D>::kPer], thr[TileRegs<D>::kPer];
};

template <int D>
__device__ __forceinline__ void tile_keys(const int* rows, const int* thrs, TileKeys<D>& tk) {
  const int key0 = threadIdx.x / TileRegs<D>::kSegs;
#pragma unroll
  for (int p = 0; p < TileRegs<D>::kPer; ++p) {
    tk.row[p] = rows[key0 + p * TileRegs<D>::kKeyStep];
    tk.thr[p] = thrs[key0 + p * TileRegs<D>::kKeyStep];
  }
}

// Stage kinds (bits 1-2 of a stage's flags): every key from the prefix source,
// every key from the suffix source (padding keys read suffix row 0), or both.
constexpr int kStagePrefix = 1, kStageSuffix = 2;

// A stage from one source (the common case) addresses its pieces as 32-bit
// byte offsets from that source's base, which stays in scalar registers; a
// stage across the prefix/suffix boundary selects a 64-bit base per piece.
template <int D>
__device__ __forceinline__ void tile_load(const AttnArgs& a, int g, int kind, const TileKeys<D>& tk,
                                          TileRegs<D>& r) {
  const int seg8 = (threadIdx.x % TileRegs<D>::kSegs) * 8;
  if (a.off32 && kind != (kStagePrefix | kStageSuffix)) {  // uniform
    const bool pre = kind == kStagePrefix;
    const uint32_t bytes = pre ? a.pre_bytes : a.suf_bytes;
    const __amdgpu_buffer_rsrc_t kr = raw_rsrc(pre ? a.kbase : a.ks, bytes);
    const __amdgpu_buffer_rsrc_t vr = raw_rsrc(pre ? a.vbase : a.vs, bytes);
    const uint32_t col = (uint32_t)(g * D + seg8) * 2u;
#pragma unroll
    for (int p = 0; p < TileRegs<D>::kPer; ++p) {
      const uint32_t off = (uint32_t)tk.row[p] + col;  // the table holds byte offsets
      r.k[p] = __builtin_amdgcn_raw_buffer_load_b128(kr, off, 0, 0);
      r.v[p] = __builtin_amdgcn_raw_buffer_load_b128(vr, off, 0, 0);
    }
    return;
  }
  const uint64_t col = (uint64_t)(g * D + seg8);
#pragma unroll
  for (int p = 0; p < TileRegs<D>::kPer; ++p) {
    // element offset of the piece: from the table's byte offset, or its row
    const uint64_t e = a.off32 ? (uint64_t)((uint32_t)tk.row[p] >> 1) + col
                               : (uint64_t)(uint32_t)tk.row[p] * (uint32_t)(a.Hkv * D) + col;
    const bool pre = tk.thr[p] == kPrefix;
    r.k[p] = *reinterpret_cast<const u32x4*>((pre ? a.kbase : a.ks) + e);
    r.v[p] = *reinterpret_cast<const u32x4*>((pre ? a.vbase : a.vs) + e);
  }
}

template <int D>
__device__ __forceinline__ void tile_store(const TileRegs<D>& r, uint16_t* lk, uint16_t* lv) {
  constexpr int kSegs = TileRegs<D>::kSegs;
#pragma unroll
  for (int p = 0; p < TileRegs<D>::kPer; ++p) {
    const int idx = threadIdx.x + p * kWaves * 64;
    const int key = idx / kSegs, seg = idx % kSegs;
    *reinterpret_cast<u32x4*>(lk + key * KLds<D>::kRow + seg * 8) = r.k[p];
    *reinterpret_cast<u32x4*>(lv + v_off<D>(key, seg)) = r.v[p];
  }
}

// Per-lane state of a wave's 32 rows.
template <int D>
struct RowState {
  f32x16 o[D / 32];  // O^T: o[db][v] holds d = 32*db + 8*(v/4) + 4*half + v%4
  float m_run;       // reference (scaled log2 units), -inf before any
  float l_run;       // sum of numerators against m_run
};

// S^T of one stage for this wave's rows: two 32-key products.
template <int D>
__device__ __forceinline__ void stage_logits(const uint16_t* lk, int kbase_off,
                                             const bf16x8 (&qf)[D / 16], f32x16 (&s)[2]) {
#pragma unroll
  for (int sub = 0; sub < 2; ++sub)
#pragma unroll
    for (int v = 0; v < 16; ++v) s[sub][v] = 0.f;
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      const bf16x8 kf = *reinterpret_cast<const bf16x8*>(
          lk + kbase_off + sub * kSub * KLds<D>::kRow + ks * 16);
      s[sub] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s[sub], 0, 0, 0);
    }
  }
}

// Logits of one stage with the keys this lane's query must not see at -inf.
template <int D>
__device__ __forceinline__ void stage_masked_logits(const uint16_t* lk, int kbase_off,
                                                    const bf16x8 (&qf)[D / 16], const int* thrs,
                                                    bool need_mask, int t, f32x16 (&s)[2]) {
  const int half = (threadIdx.x >> 5) & 1;
  stage_logits<D>(lk, kbase_off, qf, s);
  // register v of product `sub` holds key 32*sub + 16*(v/8) + 8*half + v%8:
  // runs of 8 consecutive keys, read as two 16-byte words each
  if (need_mask) {
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
#pragma unroll
      for (int v8 = 0; v8 < 2; ++v8) {
        const int* tp = thrs + kSub * sub + 16 * v8 + 8 * half;
        const int4 t0 = *reinterpret_cast<const int4*>(tp);
        const int4 t1 = *reinterpret_cast<const int4*>(tp + 4);
        const int th[8] = {t0.x, t0.y, t0.z, t0.w, t1.x, t1.y, t1.z, t1.w};
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (t < th[e]) s[sub][8 * v8 + e] = -INFINITY;
      }
  }
}

// Softmax part of one 64-key stage from the K buffer lk whose visibility
// thresholds are `thrs`: numerators into s.  The reference moves only when the stage's
// maximum exceeds it by more than kLazy (log2 units): numerators stay below
// 2^kLazy, numerator and denominator share the reference, and most stages skip
// the O rescale.
template <int D>
__device__ __forceinline__ void stage_softmax(const AttnArgs& a, const uint16_t* lk, const int* thrs,
                                              bool need_mask, int t, int kbase_off,
                                              const bf16x8 (&qf)[D / 16], RowState<D>& rs,
                                              f32x16 (&s)[2]) {
  stage_masked_logits<D>(lk, kbase_off, qf, thrs, need_mask, t, s);
  float mx = fmaxf(s[0][0], s[1][0]);
#pragma unroll
  for (int v = 1; v < 16; ++v) mx = fmaxf(mx, fmaxf(s[0][v], s[1][v]));
  mx = fmaxf(mx, partner_f(mx));
  const float mt = mx * a.c1;
  const float m_new = mt > rs.m_run + kLazy ? mt : rs.m_run;
  const float m_use = m_new == -INFINITY ? 0.f : m_new;
  const float alpha = __builtin_amdgcn_exp2f(rs.m_run - m_use);
  float sum = 0.f;
#pragma unroll
  for (int sub = 0; sub < 2; ++sub)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      s[sub][v] = __builtin_amdgcn_exp2f(fmaf(s[sub][v], a.c1, -m_use));
      sum += s[sub][v];
    }
  sum += partner_f(sum);
  rs.l_run = rs.l_run * alpha + sum;
  rs.m_run = m_new;
  if (__any(alpha != 1.f)) {
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int v = 0; v < 16; ++v) rs.o[db][v] *= alpha;
  }
}

// O^T += V^T P^T from the V buffer lv, 16 keys per product.
template <int D>
__device__ __forceinline__ void stage_pv(const uint16_t* lv, const int (&voff)[D / 32],
                                         const f32x16 (&s)[2], RowState<D>& rs) {
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) {
    bf16x8 pb[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 8; ++e) pb[kb][e] = (__bf16)s[sub][8 * kb + e];
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        s16x4 piece[2];
#pragma unroll
        for (int rd = 0; rd < 2; ++rd)
          piece[rd] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) s16x4*)(lv + voff[db] +
                                                         (sub * kSub + 16 * kb + 4 * rd) * D));
        bf16x8 vf;
        *reinterpret_cast<s16x4*>(&vf) = piece[0];
        *(reinterpret_cast<s16x4*>(&vf) + 1) = piece[1];
        rs.o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[kb], rs.o[db], 0, 0, 0);
      }
    }
  }
}

template <int D>
__global__ __launch_bounds__(kWaves * 64, 2) void attn_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t lk[2][kTile * KLds<D>::kRow];
  __shared__ __attribute__((aligned(16))) uint16_t lv[2][kTile * D];
  // key tables of the slice (rows, thresholds), then one flags word per stage:
  // bit 0 a key some row of the block must not see, bits 1-2 the stage's kind
  // (dynamic: tiles_per_split * (2 * kTile + 1) ints)
  extern __shared__ int slice_lds[];
  int* rows = slice_lds;
  int* thrs = slice_lds + a.tiles_per_split * kTile;
  int* stage_flags = slice_lds + 2 * a.tiles_per_split * kTile;

  // logical order (g, split, row block): blocks reading the same K/V tiles are
  // adjacent, hence on the same XCD and its L2
  const uint32_t L = xcd_remap(blockIdx.x, a.nblocks_padded);
  if (L >= a.nblocks) return;
  const int rb = (int)(L % a.n_row_blocks);
  const int split = (int)((L / a.n_row_blocks) % a.n_splits);
  const int g = (int)(L / ((uint32_t)a.n_splits * a.n_row_blocks));
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5;

  const int row = rb * kBlockRows + wave * kWaveRows + (lane & 31);
  const bool row_ok = row < a.R;
  const int t = row_ok ? row / a.G : -1;
  const int hi = row_ok ? row % a.G : 0;

  // keys the block's last query can see; the block's first query sees every
  // suffix key up to its own position
  const int first_t = (rb * kBlockRows) / a.G;
  const int last_row = min(a.R - 1, rb * kBlockRows + kBlockRows - 1);
  const int np_block = a.kc + (a.with_suffix ? last_row / a.G + 1 : 0);
  const int ntiles = (np_block + kTile - 1) / kTile;
  const int tile0 = split * a.tiles_per_split;
  const int nt = max(0, min(ntiles, tile0 + a.tiles_per_split) - tile0);

  // key tables of the slice, one stage per wave at a time, and whether a stage
  // has a key some row of the block must not see; all index loads first
  constexpr int kMaxIt = kMaxSliceKeys / kTile / kWaves;
  int jv[kMaxIt], sv[kMaxIt];
#pragma unroll
  for (int it = 0; it < kMaxIt; ++it) {
    const int st = wave + it * kWaves;
    jv[it] = 0;
    sv[it] = 0;
    if (st < nt) key_chunk_loads(a, (tile0 + st) * kTile + lane, jv[it], sv[it]);
  }
  // Q after the index loads: loads return in order, so the key tables (on the
  // critical path to the first K/V loads) do not wait for Q
  bf16x8 qf[D / 16];
  {
    const uint16_t* src = a.q + ((int64_t)(row_ok ? t : 0) * a.Hq + (int64_t)g * a.G + hi) * D + 8 * half;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      u32x4 v = *reinterpret_cast<const u32x4*>(src + 16 * ks);
      if (!row_ok) v = u32x4{0u, 0u, 0u, 0u};
      qf[ks] = *reinterpret_cast<bf16x8*>(&v);
    }
  }
#pragma unroll
  for (int it = 0; it < kMaxIt; ++it) {
    const int st = wave + it * kWaves;
    if (st >= nt) break;  // uniform
    const int pos = (tile0 + st) * kTile + lane;
    int krow = 0, kthr = kNever;
    if (pos < np_block) key_entry(a, pos, jv[it], sv[it], krow, kthr);
    // the row's byte offset from its source's base when every one fits in 32 bits
    rows[st * kTile + lane] = a.off32 ? (int)((uint32_t)krow * a.row_bytes) : krow;
    thrs[st * kTile + lane] = kthr;
    const uint64_t bad = __ballot(kthr > first_t), pre = __ballot(kthr == kPrefix);
    if (lane == 0)
      stage_flags[st] = (bad != 0 ? 1 : 0) | (pre != 0 ? kStagePrefix << 1 : 0) |
                        (pre != ~0ull ? kStageSuffix << 1 : 0);
  }
  __syncthreads();
  auto stage_kind = [&](int st) { return __builtin_amdgcn_readfirstlane(stage_flags[st] >> 1); };

  // per-lane LDS element offsets of the operand reads (the same for every stage)
  const int kbase_off = kappa(lane & 31) * KLds<D>::kRow + 8 * half;
  // V^T fragment pieces: lane (group g4 = (lane/16)%2, s16 = lane%16) supplies
  // row 16*kb + 8*half + 4*rd + s16/4, columns 32*db + 16*g4 + 4*(s16%4) .. +3.
  // The swizzle depends on the row modulo 4 only, so (kb, rd) add whole rows:
  // voff[db] is the offset for kb = rd = 0 and the rest are immediate offsets.
  const int s16 = lane & 15, g4 = (lane >> 4) & 1;
  int voff[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db) {
    const int vrow = 8 * half + (s16 >> 2);
    const int col = 32 * db + 16 * g4 + 4 * (s16 & 3);
    voff[db] = v_off<D>(vrow, col >> 3) + (col & 7);
  }

  RowState<D> rs;
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) rs.o[db][v] = 0.f;
  rs.m_run = -INFINITY;
  rs.l_run = 0.f;

  TileRegs<D> regs;
  TileKeys<D> tk;
  if (nt > 0) {
    tile_keys<D>(rows, thrs, tk);
    tile_load<D>(a, g, stage_kind(0), tk, regs);
    if (nt > 1) tile_keys<D>(rows + kTile, thrs + kTile, tk);
    tile_store<D>(regs, lk[0], lv[0]);
    __syncthreads();
  }
  for (int st = 0; st < nt; ++st) {
    const int cur = st & 1;
    const bool has_next = st + 1 < nt;
    // the next stage's K/V rows load during this stage; the table entries of
    // the stage after it are read now, for the next iteration
    if (has_next) {
      tile_load<D>(a, g, stage_kind(st + 1), tk, regs);
      if (st + 2 < nt) tile_keys<D>(rows + (st + 2) * kTile, thrs + (st + 2) * kTile, tk);
    }
    f32x16 s[2];
    stage_softmax<D>(a, lk[cur], thrs + st * kTile, stage_flags[st] & 1, t, kbase_off, qf, rs, s);
    stage_pv<D>(lv[cur], voff, s, rs);
    if (has_next) {
      tile_store<D>(regs, lk[cur ^ 1], lv[cur ^ 1]);
      __syncthreads();
    }
  }

  // Output rows through LDS, so that every global store is a whole 16-byte
  // piece of a row and 16 lanes cover a row: the wave's 32 rows (O/l in
  // bf16) go to its own slice of the K stage buffer, which every wave has
  // finished reading after this barrier.
  __syncthreads();
  {
    constexpr int kRow = KLds<D>::kRow;
    uint16_t* tile = reinterpret_cast<uint16_t*>(lk) + wave * kWaveRows * kRow;
    const float inv = rs.l_run > 0.f ? 1.f / rs.l_run : 0.f;
    // o[db][v] holds d = 32*db + 8*(v/4) + 4*half + v%4 of this lane's row
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        __bf16 b[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) b[j] = (__bf16)(rs.o[db][4 * q4 + j] * inv);
        *reinterpret_cast<uint2*>(tile + (lane & 31) * kRow + 32 * db + 8 * q4 + 4 * half) =
            *reinterpret_cast<uint2*>(b);
      }
    __builtin_amdgcn_wave_barrier();
    constexpr int kSegs = D / 8, kRowsPerPass = 64 / kSegs;
    const int seg = lane % kSegs;
    const int row_base = rb * kBlockRows + wave * kWaveRows;
#pragma unroll
    for (int r0 = 0; r0 < kWaveRows; r0 += kRowsPerPass) {
      const int rr = r0 + lane / kSegs;
      const int orow = row_base + rr;
      const uint4 v = *reinterpret_cast<const uint4*>(tile + rr * kRow + seg * 8);
      if (orow < a.R) {
        uint16_t* dst;
        if (!a.partial)
          dst = a.out + ((int64_t)(orow / a.G) * a.Hq + (int64_t)g * a.G + orow % a.G) * D;
        else
          dst = a.o_part + (((int64_t)split * a.Hkv + g) * a.R + orow) * D;
        *reinterpret_cast<uint4*>(dst + seg * 8) = v;
      }
    }
  }
  // the reference the numerators were taken against (0 while no key was seen)
  if (a.partial && row_ok && half == 0)
    a.ml_part[((int64_t)split * a.Hkv + g) * a.R + row] =
        make_float2(rs.m_run == -INFINITY ? 0.f : rs.m_run, rs.l_run);
}

// Merges the splits of each row in split order: out = sum_s w_s Ohat_s with
// w_s = e_s l_s / sum_s e_s l_s, e_s = exp2(m_s - max m), Ohat_s = O_s / l_s,
// as a running merge over batches of kCombineBatch splits whose loads are in
// flight together.  One thread per (row, 8 columns).
constexpr int kCombineBatch = 8;

template <int D>
__global__ __launch_bounds__(256) void combine_kernel(const uint16_t* __restrict__ o_part,
                                                      const float2* __restrict__ ml_part,
                                                      uint16_t* __restrict__ out, int n_splits,
                                                      int Hkv, int R, int G, int Hq) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t rows = (int64_t)Hkv * R;
  if (idx >= rows * (D / 8)) return;
  const int64_t grow = idx / (D / 8);
  const int c8 = (int)(idx % (D / 8)) * 8;
  float M = -INFINITY, Lsum = 0.f;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < n_splits; s0 += kCombineBatch) {
    // unconditional loads (a split past the last re-reads the last one and is
    // then ignored), so the whole batch is in flight together
    float2 ml[kCombineBatch];
    uint4 raw[kCombineBatch];
#pragma unroll
    for (int i = 0; i < kCombineBatch; ++i) {
      const int64_t sp = min(s0 + i, n_splits - 1);
      ml[i] = ml_part[sp * rows + grow];
      raw[i] = *reinterpret_cast<const uint4*>(o_part + (sp * rows + grow) * D + c8);
    }
#pragma unroll
    for (int i = 0; i < kCombineBatch; ++i)
      if (s0 + i >= n_splits) ml[i] = make_float2(0.f, 0.f);
#pragma unroll
    for (int i = 0; i < kCombineBatch; ++i) {
      if (!(ml[i].y > 0.f)) continue;  // absent, or the split saw no key of this row
      if (ml[i].x > M) {
        const float scale = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(M - ml[i].x);
        Lsum *= scale;
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] *= scale;
        M = ml[i].x;
      }
      const float wgt = __builtin_amdgcn_exp2f(ml[i].x - M) * ml[i].y;
      Lsum += wgt;
      const __bf16* h = reinterpret_cast<const __bf16*>(&raw[i]);
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] += wgt * (float)h[j];
    }
  }
  const int g = (int)(grow / R), row = (int)(grow % R);
  const int t = row / G, i = row % G;
  const float inv = 1.f / Lsum;
  __bf16 b[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) b[j] = (__bf16)(acc[j] * inv);
  *reinterpret_cast<uint4*>(out + ((int64_t)t * Hq + (int64_t)g * G + i) * D + c8) =
      *reinterpret_cast<uint4*>(b);
}

// ---------------------------------------------------------------------------
// fp32 path: one wave per (query t, head h).  Lane l visits keys l, l+64, ...
// of the row's key sequence with its own online softmax (fp32, exp2 with the
// scale folded in), then the 64 lane states are merged by a butterfly.
// ---------------------------------------------------------------------------
struct AttnArgsF32 {
  const float* q;
  const float* kbase;
  const float* vbase;
  int64_t chunk_stride;
  const int32_t* chunk_off;
  int32_t direct;
  const int32_t* sel;
  int64_t kc, n;
  int c;
  const float* ks;
  const float* vs;
  float* out;
  int S, Hq, Hkv, G;
  float c1;
};

template <int D>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgsF32 a) {
  const int64_t rid = blockIdx.x;  // t * Hq + h
  const int t = (int)(rid / a.Hq), h = (int)(rid % a.Hq), g = h / a.G;
  const int lane = threadIdx.x;
  const float* qr = a.q + rid * D;
  float o[D];
#pragma unroll
  for (int e = 0; e < D; ++e) o[e] = 0.f;
  float m = -INFINITY, l = 0.f;
  const int64_t np = a.kc + t + 1;
  for (int64_t pos = lane; pos < np; pos += 64) {
    const float* kr;
    const float* vr;
    if (pos < a.kc) {
      const int64_t u = pos / a.c;
      const int off = (int)(pos - u * a.c);
      const int64_t j = a.sel[u];
      if (j < 0 || off >= min<int64_t>(a.c, a.n - j * a.c)) continue;
      const int64_t slot = a.chunk_off ? (int64_t)a.chunk_off[u] : (a.direct ? j : u);
      const int64_t e = slot * a.chunk_stride + ((int64_t)off * a.Hkv + g) * D;
      kr = a.kbase + e;
      vr = a.vbase + e;
    } else {
      const int64_t e = ((pos - a.kc) * a.Hkv + g) * D;
      kr = a.ks + e;
      vr = a.vs + e;
    }
    float dot = 0.f;
#pragma unroll
    for (int e = 0; e < D; ++e) dot = fmaf(qr[e], kr[e], dot);
    const float s = dot * a.c1;
    const float mn = fmaxf(m, s);
    const float alpha = __builtin_amdgcn_exp2f(m - mn);
    const float p = __builtin_amdgcn_exp2f(s - mn);
    l = l * alpha + p;
#pragma unroll
    for (int e = 0; e < D; ++e) o[e] = fmaf(p, vr[e], o[e] * alpha);
    m = mn;
  }
  // merge of the 64 lanes' (m, l, o) through LDS: the wave's maximum
  // reference, each lane's scale, then lane e sums element e over the lanes
  __shared__ float so[64][D + 1];  // padded: lane j's row starts one bank later
  __shared__ float sa[64];
#pragma unroll
  for (int e = 0; e < D; ++e) so[lane][e] = o[e];
  float M = m;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) M = fmaxf(M, __shfl_xor(M, off));
  const float scale = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - M);
  float L = l * scale;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) L += __shfl_xor(L, off);
  sa[lane] = scale;
  __syncthreads();
  const float inv = L > 0.f ? 1.f / L : 0.f;
  float* dst = a.out + rid * D;
  for (int e = lane; e < D; e += 64) {
    float acc = 0.f;
    for (int j = 0; j < 64; ++j) acc = fmaf(so[j][e], sa[j], acc);
    dst[e] = acc * inv;
  }
}

}  // namespace

AttnPlan make_attn_plan(const ckv_dims* d, int64_t k, bool with_suffix) {
  AttnPlan p{};
  const int G = d->n_q_heads / d->n_kv_heads;
  p.rows = G * d->n_suffix;
  if (d->dtype == CKV_DTYPE_F32) {  // one wave per row, no splits
    p.n_splits = 1;
    return p;
  }
  const int64_t np = k * d->chunk_size + (with_suffix ? d->n_suffix : 0);
  const int64_t ntiles = std::max<int64_t>(1, ceil_div(np, kTile));  // no keys: one empty split
  const int64_t base = (int64_t)d->n_kv_heads * ceil_div(p.rows, kBlockRows);
  // at most ~2 workgroups per CU, keeping >= 4 stages per split and no more
  // keys per split than the workgroup's code table holds; then the fewest
  // splits that give the same stages per split
  int64_t splits = std::max<int64_t>(1, 512 / base);
  splits = std::min<int64_t>(splits, std::max<int64_t>(1, ntiles / 4));
  splits = std::max<int64_t>(splits, ceil_div(ntiles, kMaxSliceKeys / kTile));
  splits = ceil_div(ntiles, ceil_div(ntiles, splits));
  p.n_splits = (int32_t)splits;
  size_t off = 0;
  if (splits > 1) {
    const size_t rows = (size_t)d->n_kv_heads * p.rows;
    p.off_o = off;
    off = align_up(off + (size_t)splits * rows * d->head_dim * sizeof(uint16_t), 256);
    p.off_ml = off;
    off = align_up(off + (size_t)splits * rows * sizeof(float2), 256);
  }
  p.bytes = off;
  return p;
}

namespace {

// Arguments of one bf16 attention launch over the kept chunks sel[0..k) of
// src (and the suffix when with_suffix) in n_splits key splits.
ckv_status attn_args(const ckv_dims* d, const void* q, const ChunkSource& src, const int32_t* sel,
                     int64_t k, const void* k_suffix, const void* v_suffix, bool with_suffix,
                     int32_t n_splits, AttnArgs& a) {
  a.q = static_cast<const uint16_t*>(q);
  a.kbase = static_cast<const uint16_t*>(src.k_base);
  a.vbase = static_cast<const uint16_t*>(src.v_base);
  a.chunk_off = src.chunk_off;
  a.direct = src.direct;
  {
    const int64_t hd = (int64_t)d->n_kv_heads * d->head_dim;
    if (src.chunk_stride % hd != 0) CKV_FAIL(CKV_EINVAL, "chunk stride is not a whole number of rows");
    const int64_t rps = src.chunk_stride / hd;
    // largest source row a key can name: every slot index is below n_slots
    if (src.n_slots < 0 || src.n_slots * rps >= (int64_t(1) << 31))
      CKV_FAIL(CKV_EUNSUPPORTED, "chunk source too large");
    a.rows_per_slot = (int)rps;
    // 32-bit byte offsets reach every row of both sources
    const int64_t rb = hd * (int64_t)sizeof(uint16_t);
    a.row_bytes = (uint32_t)rb;
    // (strictly below 4 GiB, so each source's byte count is a buffer size)
    const int64_t pre = src.n_slots * rps * rb, suf = (int64_t)d->n_suffix * rb;
    a.off32 = pre < (int64_t(1) << 32) && suf < (int64_t(1) << 32) &&
              g_force_wide.load(std::memory_order_relaxed) == 0;
    a.pre_bytes = (uint32_t)std::min<int64_t>(pre, UINT32_MAX);
    a.suf_bytes = (uint32_t)std::min<int64_t>(suf, UINT32_MAX);
  }
  a.sel = sel;
  a.kc = (int)(k * d->chunk_size);
  a.n = d->n_prefix;
  a.m = ceil_div(d->n_prefix, d->chunk_size);
  a.c = d->chunk_size;
  a.log2c = (d->chunk_size & (d->chunk_size - 1)) == 0 ? __builtin_ctz(d->chunk_size) : -1;
  a.ks = static_cast<const uint16_t*>(k_suffix);
  a.vs = static_cast<const uint16_t*>(v_suffix);
  a.S = d->n_suffix; a.Hq = d->n_q_heads; a.Hkv = d->n_kv_heads;
  a.G = d->n_q_heads / d->n_kv_heads; a.R = a.G * d->n_suffix;
  a.n_splits = n_splits;
  a.with_suffix = with_suffix ? 1 : 0;
  const int64_t ntiles = ceil_div(a.kc + (with_suffix ? a.S : 0), kTile);
  a.tiles_per_split = (int)ceil_div(ntiles, n_splits);  // <= kMaxSliceKeys / kTile
  a.n_row_blocks = (int)ceil_div(a.R, kBlockRows);
  a.c1 = resolve_scale(d) * 1.4426950408889634f;
  a.nblocks = (uint32_t)((int64_t)a.Hkv * a.n_row_blocks * a.n_splits);
  a.nblocks_padded = (uint32_t)align_up(a.nblocks, 8);
  return CKV_OK;
}

ckv_status launch_attn_kernel(const ckv_dims* d, const AttnArgs& a, hipStream_t st) {
  const size_t slice_bytes = (size_t)a.tiles_per_split * (2 * kTile + 1) * sizeof(int);
  if (d->head_dim == 128)
    hipLaunchKernelGGL(attn_kernel<128>, dim3(a.nblocks_padded), dim3(kWaves * 64), slice_bytes, st, a);
  else
    hipLaunchKernelGGL(attn_kernel<64>, dim3(a.nblocks_padded), dim3(kWaves * 64), slice_bytes, st, a);
  CKV_HIP(hipGetLastError());
  return CKV_OK;
}

ckv_status launch_combine(const ckv_dims* d, const uint16_t* o_part, const float2* ml_part,
                          int32_t n_splits, void* out, hipStream_t st) {
  const int G = d->n_q_heads / d->n_kv_heads, R = G * d->n_suffix;
  const int64_t work = (int64_t)d->n_kv_heads * R * (d->head_dim / 8);
  uint16_t* o = static_cast<uint16_t*>(out);
  if (d->head_dim == 128)
    hipLaunchKernelGGL(combine_kernel<128>, dim3((unsigned)ceil_div(work, 256)), dim3(256), 0, st,
                       o_part, ml_part, o, n_splits, d->n_kv_heads, R, G, d->n_q_heads);
  else
    hipLaunchKernelGGL(combine_kernel<64>, dim3((unsigned)ceil_div(work, 256)), dim3(256), 0, st,
                       o_part, ml_part, o, n_splits, d->n_kv_heads, R, G, d->n_q_heads);
  CKV_HIP(hipGetLastError());
  return CKV_OK;
}

// Split partials of a parted attention: splits [0, max_splits) of o_part
// ([split][Hkv][R][D] bf16) then of ml_part ([split][Hkv][R] float2).
size_t part_o_bytes(const ckv_dims* d, int64_t max_splits) {
  const int G = d->n_q_heads / d->n_kv_heads;
  return align_up((size_t)max_splits * d->n_kv_heads * G * d->n_suffix * d->head_dim *
                      sizeof(uint16_t), 256);
}

}  // namespace

ckv_status launch_attn(const ckv_dims* d, const void* q, const ChunkSource& src, const int32_t* sel,
                       int64_t k, const void* k_suffix, const void* v_suffix, void* out, void* ws,
                       size_t ws_bytes, hipStream_t st) {
  if (d->dtype == CKV_DTYPE_F32) {
    AttnArgsF32 a;
    a.q = static_cast<const float*>(q);
    a.kbase = static_cast<const float*>(src.k_base);
    a.vbase = static_cast<const float*>(src.v_base);
    a.chunk_stride = src.chunk_stride;
    a.chunk_off = src.chunk_off;
    a.direct = src.direct;
    a.sel = sel;
    a.kc = k * d->chunk_size;
    a.n = d->n_prefix;
    a.c = d->chunk_size;
    a.ks = static_cast<const float*>(k_suffix);
    a.vs = static_cast<const float*>(v_suffix);
    a.out = static_cast<float*>(out);
    a.S = d->n_suffix; a.Hq = d->n_q_heads; a.Hkv = d->n_kv_heads;
    a.G = d->n_q_heads / d->n_kv_heads;
    a.c1 = resolve_scale(d) * 1.4426950408889634f;
    hipLaunchKernelGGL(attn_f32_kernel<64>, dim3((unsigned)((int64_t)a.S * a.Hq)), dim3(64), 0, st, a);
    CKV_HIP(hipGetLastError());
    return CKV_OK;
  }
  const AttnPlan p = make_attn_plan(d, k);
  if (ws_bytes < p.bytes) CKV_FAIL(CKV_EINVAL, "attention workspace too small: %zu < %zu", ws_bytes, p.bytes);
  AttnArgs a;
  ckv_status s = attn_args(d, q, src, sel, k, k_suffix, v_suffix, true, p.n_splits, a);
  if (s != CKV_OK) return s;
  a.out = static_cast<uint16_t*>(out);
  a.partial = p.n_splits > 1 ? 1 : 0;
  a.o_part = a.partial ? reinterpret_cast<uint16_t*>(static_cast<char*>(ws) + p.off_o) : nullptr;
  a.ml_part = a.partial ? reinterpret_cast<float2*>(static_cast<char*>(ws) + p.off_ml) : nullptr;
  if ((s = launch_attn_kernel(d, a, st)) != CKV_OK) return s;
  if (a.partial) return launch_combine(d, a.o_part, a.ml_part, a.n_splits, out, st);
  return CKV_OK;
}

// Every share holds one chunk plus a part of the rest that shrinks
// geometrically, share j weighing kShareA^j kShareB^(parts-1-j), so that the
// last share -- whose attention is all that follows the last copy -- is the
// smallest and no share is empty (integer arithmetic: the same shares on every
// host).  1 <= parts <= n_late.
constexpr int64_t kShareA = 1, kShareB = 2;

int64_t attn_late_part_begin(int64_t n_late, int parts, int i) {
  int64_t cum = 0, total = 0;
  for (int j = 0; j < parts; ++j) {
    int64_t w = 1;
    for (int e = 0; e < j; ++e) w *= kShareA;
    for (int e = 0; e < parts - 1 - j; ++e) w *= kShareB;
    if (j < i) cum += w;
    total += w;
  }
  return i + (n_late - parts) * cum / total;
}

int64_t attn_parted_splits(const ckv_dims* d, int64_t k, int max_late_parts) {
  int64_t most = 0;
  for (int64_t ka = 0; ka <= k; ++ka) {
    const int64_t nl = k - ka;
    const int parts = (int)std::min<int64_t>(max_late_parts, nl);
    int64_t n = make_attn_plan(d, ka, true).n_splits;
    for (int i = 0; i < parts; ++i)
      n += make_attn_plan(d, attn_late_part_begin(nl, parts, i + 1) -
                                 attn_late_part_begin(nl, parts, i), false).n_splits;
    most = std::max(most, n);
  }
  return most;
}

size_t attn_parted_bytes(const ckv_dims* d, int64_t max_splits) {
  const int G = d->n_q_heads / d->n_kv_heads;
  return align_up(part_o_bytes(d, max_splits) +
                      (size_t)max_splits * d->n_kv_heads * G * d->n_suffix * sizeof(float2),
                  256);
}

ckv_status launch_attn_part(const ckv_dims* d, const void* q, const ChunkSource& src,
                            const int32_t* sel, int64_t k, const void* k_suffix,
                            const void* v_suffix, bool with_suffix, void* ws, int64_t max_splits,
                            int32_t split_base, int32_t* n_splits, hipStream_t st) {
  if (d->dtype != CKV_DTYPE_BF16) CKV_FAIL(CKV_EUNSUPPORTED, "parted attention is bf16 only");
  if (k == 0 && !with_suffix) CKV_FAIL(CKV_EINVAL, "an attention part without the suffix needs chunks");
  const AttnPlan p = make_attn_plan(d, k, with_suffix);
  if (split_base < 0 || split_base + (int64_t)p.n_splits > max_splits)
    CKV_FAIL(CKV_EINVAL, "attention splits %d + %d exceed the workspace's %lld", split_base,
             p.n_splits, (long long)max_splits);
  AttnArgs a;
  ckv_status s = attn_args(d, q, src, sel, k, k_suffix, v_suffix, with_suffix, p.n_splits, a);
  if (s != CKV_OK) return s;
  const size_t rows = (size_t)d->n_kv_heads * a.R;
  a.out = nullptr;
  a.partial = 1;
  a.o_part = static_cast<uint16_t*>(ws) + (size_t)split_base * rows * d->head_dim;
  a.ml_part = reinterpret_cast<float2*>(static_cast<char*>(ws) + part_o_bytes(d, max_splits)) +
              (size_t)split_base * rows;
  *n_splits = p.n_splits;
  return launch_attn_kernel(d, a, st);
}

ckv_status launch_attn_combine(const ckv_dims* d, const void* ws, int64_t max_splits,
                               int32_t n_splits, void* out, hipStream_t st) {
  if (n_splits < 1 || n_splits > max_splits)
    CKV_FAIL(CKV_EINVAL, "combine of %d splits (workspace holds %lld)", n_splits,
             (long long)max_splits);
  return launch_combine(d, static_cast<const uint16_t*>(ws),
                        reinterpret_cast<const float2*>(static_cast<const char*>(ws) +
                                                        part_o_bytes(d, max_splits)),
                        n_splits, out, st);
}

}  // namespace ckv

extern "C" ckv_status ckv_debug_attn_wide_addressing(int32_t force_wide) {
  ckv::clear_error();
  if (force_wide != 0 && force_wide != 1) CKV_FAIL(CKV_EINVAL, "force_wide must be 0 or 1");
  ckv::g_force_wide.store(force_wide, std::memory_order_relaxed);
  return CKV_OK;
}
