// attn.hip -- Re-Prefill sparse attention (Def. 2.1) for gfx950, bf16.
//
// For query t of head h (KV head g = h / G) the keys are the tokens of the k
// kept chunks (compact positions 0 .. k*c-1; rows past n of a short last chunk
// are masked) followed by the suffix tokens 0..t (causal).
//
// Rows of one KV head are r = t*G + i (query t, head g*G + i), so the G query
// heads that share a KV head share every K/V tile.  A workgroup owns 128 rows
// (4 waves x 32) and one contiguous slice ("split") of the key positions.  Per
// 64-key stage:
//   S^T = K Q^T   bf16 MFMA 32x32x16, A = K rows from LDS, B = Q^T in
//                 registers: every lane owns one query row and 16 keys;
//   online softmax in fp32 (exp2 with sm_scale*log2 e folded in) with a lazy
//                 reference: it moves only when a stage's maximum exceeds it
//                 by more than 2^8, so most stages skip the O rescale;
//   O^T += V^T P^T  A = V^T read from LDS with the transposing
//                 ds_read_tr16_b64, B = P^T straight from the softmax registers.
// The K operand rows are loaded in a permuted order so that the registers a
// lane holds after the first product are exactly the 8 consecutive keys the
// second product needs from it -- no register shuffles between the two.
// Splits write their normalised partial output O/l in bf16 (the output's own
// type and range) plus (reference, l) in fp32; a combine kernel merges them in
// split order (deterministic).

#include "ckv_internal.h"

namespace ckv {
namespace {

constexpr int kWaves = 4;
constexpr int kWaveRows = 32;
constexpr int kBlockRows = kWaves * kWaveRows;  // 128
constexpr int kTile = 64;  // keys per LDS stage
constexpr int kSub = 32;   // keys per MFMA product
constexpr int kNoKey = 0x7fffffff;  // visibility limit of a masked key
constexpr float kLazy = 8.f;        // headroom of the lazy softmax reference (log2 units)

// MFMA row p of the K operand holds key kappa(p); afterwards register v of a
// lane in half h holds key 16*(v/8) + 8*h + v%8.
__device__ __forceinline__ int kappa(int p) {
  const int i = p >> 3, h = (p >> 2) & 1, j = p & 3;
  return 16 * (i >> 1) + 8 * h + 4 * (i & 1) + j;
}

// LDS swizzles (XOR of 16-byte segment index), conflict-free for the access
// patterns of the two operand reads.
template <int D>
__device__ __forceinline__ int k_swz(int row) {
  if constexpr (D == 128)
    return ((row & 1) ? 1 : 0) ^ ((row & 2) ? 2 : 0) ^ ((row & 4) ? 8 : 0) ^ ((row & 8) ? 4 : 0);
  else
    return ((row & 1) ? 1 : 0) ^ ((row & 2) ? 2 : 0) ^ ((row & 4) ? 1 : 0) ^ ((row & 8) ? 4 : 0);
}
template <int D>
__device__ __forceinline__ int v_swz(int row) {
  if constexpr (D == 128)
    return ((row & 1) ? 4 : 0) ^ ((row & 2) ? 10 : 0);
  else
    return ((row & 1) ? 2 : 0) ^ ((row & 2) ? 4 : 0);
}
template <int D>
__device__ __forceinline__ int k_off(int row, int seg) { return row * D + ((seg ^ k_swz<D>(row)) << 3); }
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
  int64_t chunk_stride;    // elements
  const int32_t* chunk_off;
  int32_t direct;
  const int32_t* sel;      // [k]
  int kc;                  // k * c prefix positions (< 2^31)
  int64_t n;
  int c;
  int log2c;               // log2(c) when c is a power of two, else -1
  int short_tail;          // c - n % c when the last chunk is short, else 0
  const uint16_t* ks;      // [S][Hkv][D]
  const uint16_t* vs;
  uint16_t* out;           // [S][Hq][D]
  uint16_t* o_part;        // [splits][Hkv][R][D]: O / l, bf16
  float2* ml_part;         // [splits][Hkv][R]
  int S, Hq, Hkv, G, R, n_splits, tiles_per_split, n_row_blocks;
  float c1;
  uint32_t nblocks, nblocks_padded;
};

// The K/V rows of one 64-key stage, fetched into registers (while the previous
// stage is consumed from LDS) and then written to the other LDS buffer.
template <int D>
struct TileRegs {
  static constexpr int kPer = kTile * (D / 8) / (kWaves * 64);  // 16-byte pieces per thread
  u32x4 k[kPer], v[kPer];
  int lim[kPer];
};

// Chunk index (and slot-table entry) of each piece's key, fetched one stage
// ahead of its K/V rows so that the row loads never wait on the index loads.
// The loads are unconditional (clamped to the last kept chunk) and their values
// are only interpreted by tile_load.
template <int D>
struct TileIdx {
  int32_t j[TileRegs<D>::kPer];     // sel[u] of the piece's chunk u
  int32_t slot[TileRegs<D>::kPer];  // chunk_off[u] when a slot table is used
};

// Kept chunk u holding compact position pos.  A power-of-two c uses a shift;
// any other supported c is a multiple of 64 or 32, and u is then computed per
// piece with a 32-bit division.
__device__ __forceinline__ int chunk_of(const AttnArgs& a, int pos) {
  return a.log2c >= 0 ? (pos >> a.log2c) : (int)((uint32_t)pos / (uint32_t)a.c);
}

template <int D>
__device__ __forceinline__ void tile_index(const AttnArgs& a, int tile, TileIdx<D>& x) {
  constexpr int kSegs = D / 8;
  if (a.kc == 0) return;
  const int pos0 = tile * kTile;
  const int last = a.kc / a.c - 1;
#pragma unroll
  for (int p = 0; p < TileRegs<D>::kPer; ++p) {
    const int key = (threadIdx.x + p * kWaves * 64) / kSegs;
    const int u = min(chunk_of(a, pos0 + key), last);
    x.j[p] = a.sel[u];
    if (a.chunk_off) x.slot[p] = a.chunk_off[u];
  }
}

// Fetches stage `tile` of key positions and each key's visibility limit (a row
// with query t sees the key iff t >= lim).  Loads are unconditional: a masked
// key reads suffix row 0 of this KV head instead (finite data; its probability
// is forced to zero, so it contributes nothing).
template <int D>
__device__ __forceinline__ void tile_load(const AttnArgs& a, int g, int tile, const TileIdx<D>& x,
                                          TileRegs<D>& r) {
  constexpr int kSegs = D / 8;
  const int pos0 = tile * kTile;
#pragma unroll
  for (int p = 0; p < TileRegs<D>::kPer; ++p) {
    const int idx = threadIdx.x + p * kWaves * 64;
    const int key = idx / kSegs, seg = idx % kSegs;
    const int pos = pos0 + key;
    const int col = g * D + seg * 8;
    const uint16_t* ksrc = a.ks + col;
    const uint16_t* vsrc = a.vs + col;
    int limit = kNoKey;
    if (pos < a.kc) {
      const int u = chunk_of(a, pos);
      const int off = pos - u * a.c;
      const int j = x.j[p];
      const int len = j >= 0 ? (int)min<int64_t>(a.c, a.n - (int64_t)j * a.c) : 0;  // outside [0, m): empty
      if (off < len) {
        const int slot = a.chunk_off ? x.slot[p] : (a.direct ? j : u);
        const int64_t e = (int64_t)slot * a.chunk_stride + (off * a.Hkv * D + col);
        ksrc = a.kbase + e;
        vsrc = a.vbase + e;
        limit = -1;
      }
    } else if (pos < a.kc + a.S) {
      const int tok = pos - a.kc;
      ksrc += tok * a.Hkv * D;
      vsrc += tok * a.Hkv * D;
      limit = tok;
    }
    r.k[p] = *reinterpret_cast<const u32x4*>(ksrc);
    r.v[p] = *reinterpret_cast<const u32x4*>(vsrc);
    r.lim[p] = limit;
  }
}

template <int D>
__device__ __forceinline__ void tile_store(const TileRegs<D>& r, uint16_t* lk, uint16_t* lv, int* lim) {
  constexpr int kSegs = D / 8;
#pragma unroll
  for (int p = 0; p < TileRegs<D>::kPer; ++p) {
    const int idx = threadIdx.x + p * kWaves * 64;
    const int key = idx / kSegs, seg = idx % kSegs;
    *reinterpret_cast<u32x4*>(lk + k_off<D>(key, seg)) = r.k[p];
    *reinterpret_cast<u32x4*>(lv + v_off<D>(key, seg)) = r.v[p];
    if (seg == 0) lim[key] = r.lim[p];
  }
}

template <int D>
__global__ __launch_bounds__(kWaves * 64, 2) void attn_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t lk[2][kTile * D];
  __shared__ __attribute__((aligned(16))) uint16_t lv[2][kTile * D];
  __shared__ int lim[2][kTile];

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

  // last query of the block bounds the suffix keys anyone here can see
  const int first_t = (rb * kBlockRows) / a.G;
  const int last_row = min(a.R - 1, rb * kBlockRows + kBlockRows - 1);
  const int np_block = a.kc + last_row / a.G + 1;
  const int ntiles = (np_block + kTile - 1) / kTile;
  const int tile0 = split * a.tiles_per_split;
  const int tile1 = min(ntiles, tile0 + a.tiles_per_split);
  // prefix positions before vis_end are real tokens whatever chunks were kept
  const int vis_end = a.kc - a.short_tail;

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

  // per-lane LDS element offsets of the operand reads (the same for every stage)
  const int krow = kappa(lane & 31);
  int koff[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) koff[ks] = k_off<D>(krow, 2 * ks + half);
  const int s16 = lane & 15, g4 = (lane >> 4) & 1;
  int voff[D / 32][2][2];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int rd = 0; rd < 2; ++rd) {
        // V^T fragment piece: lane (group g4 = (lane/16)%2, s16 = lane%16) supplies
        // row 16*kb + 8*half + 4*rd + s16/4, columns 32*db + 16*g4 + 4*(s16%4) .. +3
        const int vrow = 16 * kb + 8 * half + 4 * rd + (s16 >> 2);
        const int col = 32 * db + 16 * g4 + 4 * (s16 & 3);
        voff[db][kb][rd] = v_off<D>(vrow, col >> 3) + (col & 7);
      }

  f32x16 o[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[db][v] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  TileRegs<D> regs;
  TileIdx<D> idx_next;
  if (tile0 < tile1) {
    TileIdx<D> idx0;
    tile_index<D>(a, tile0, idx0);
    tile_load<D>(a, g, tile0, idx0, regs);
    if (tile0 + 1 < tile1) tile_index<D>(a, tile0 + 1, idx_next);
    tile_store<D>(regs, lk[0], lv[0], lim[0]);
    __syncthreads();
  }
  for (int tile = tile0; tile < tile1; ++tile) {
    const int cur = (tile - tile0) & 1;
    const bool has_next = tile + 1 < tile1;
    if (has_next) {
      tile_load<D>(a, g, tile + 1, idx_next, regs);
      if (tile + 2 < tile1) tile_index<D>(a, tile + 2, idx_next);
    }
    // no key of this stage needs a mask for any row of the block when it ends
    // before the kept prefix's possibly short tail, or when its suffix keys are
    // seen by the block's first query and its prefix keys are all real tokens
    const int pos0 = tile * kTile, pos_end = pos0 + kTile;
    const bool all_vis = pos_end <= vis_end ||
                         (pos_end <= a.kc + first_t + 1 && (pos0 >= a.kc || a.short_tail == 0));

    // S^T for the two 32-key halves: two independent MFMA chains
    f32x16 s[2];
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
#pragma unroll
      for (int v = 0; v < 16; ++v) s[sub][v] = 0.f;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
        bf16x8 kf = *reinterpret_cast<const bf16x8*>(&lk[cur][sub * kSub * D + koff[ks]]);
        s[sub] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s[sub], 0, 0, 0);
      }
    }
    // register v of half `sub` holds key 32*sub + 16*(v/8) + 8*half + v%8
    if (!all_vis) {
#pragma unroll
      for (int sub = 0; sub < 2; ++sub)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = kSub * sub + 16 * (v >> 3) + 8 * half + (v & 7);
          if (t < lim[cur][key]) s[sub][v] = -INFINITY;
        }
    }
    float mx = fmaxf(s[0][0], s[1][0]);
#pragma unroll
    for (int v = 1; v < 16; ++v) mx = fmaxf(mx, fmaxf(s[0][v], s[1][v]));
    mx = fmaxf(mx, partner_f(mx));
    // The reference m_run only moves when the stage's maximum exceeds it by more
    // than kLazy (log2 units): weights stay below 2^kLazy, numerator and
    // denominator share the reference, and most stages skip the O rescale.
    const float mt = mx * a.c1;
    const float m_new = mt > m_run + kLazy ? mt : m_run;
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
    float rs = 0.f;
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        s[sub][v] = __builtin_amdgcn_exp2f(fmaf(s[sub][v], a.c1, -m_use));
        rs += s[sub][v];
      }
    rs += partner_f(rs);
    l_run = l_run * alpha + rs;
    m_run = m_new;
    if (__any(alpha != 1.f)) {
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[db][v] *= alpha;
    }

    // O^T += V^T P^T, 16 keys per product
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
                (__attribute__((address_space(3))) s16x4*)(&lv[cur][sub * kSub * D + voff[db][kb][rd]]));
          bf16x8 vf;
          *reinterpret_cast<s16x4*>(&vf) = piece[0];
          *(reinterpret_cast<s16x4*>(&vf) + 1) = piece[1];
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[kb], o[db], 0, 0, 0);
        }
      }
    }
    if (has_next) {
      tile_store<D>(regs, lk[cur ^ 1], lv[cur ^ 1], lim[cur ^ 1]);
      __syncthreads();
    }
  }

  // o[db][v] holds d = 32*db + 8*(v/4) + 4*half + v%4 of this lane's row
  if (!row_ok) return;
  if (a.n_splits == 1) {
    const float inv = 1.f / l_run;
    uint16_t* dst = a.out + ((int64_t)t * a.Hq + (int64_t)g * a.G + hi) * D + 4 * half;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        __bf16 b[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) b[j] = (__bf16)(o[db][4 * q4 + j] * inv);
        *reinterpret_cast<uint2*>(dst + 32 * db + 8 * q4) = *reinterpret_cast<uint2*>(b);
      }
  } else {
    const int64_t prow = ((int64_t)split * a.Hkv + g) * a.R + row;
    uint16_t* dst = a.o_part + prow * D + 4 * half;
    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        __bf16 b[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) b[j] = (__bf16)(o[db][4 * q4 + j] * inv);
        *reinterpret_cast<uint2*>(dst + 32 * db + 8 * q4) = *reinterpret_cast<uint2*>(b);
      }
    // the reference the numerators were taken against (0 while no key was seen)
    if (half == 0) a.ml_part[prow] = make_float2(m_run == -INFINITY ? 0.f : m_run, l_run);
  }
}

// Merges the splits of each row in split order: out = sum_s w_s Ohat_s with
// w_s = e_s l_s / sum_s e_s l_s, e_s = exp2(m_s - max m), Ohat_s = O_s / l_s.
// One thread per (row, 8 columns).
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
  float M = -INFINITY;
  for (int s = 0; s < n_splits; ++s) {
    const float2 ml = ml_part[s * rows + grow];
    if (ml.y > 0.f) M = fmaxf(M, ml.x);
  }
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float Lsum = 0.f;
  for (int s = 0; s < n_splits; ++s) {
    const float2 ml = ml_part[s * rows + grow];
    if (!(ml.y > 0.f)) continue;  // the split saw no key of this row
    const float wgt = __builtin_amdgcn_exp2f(ml.x - M) * ml.y;
    Lsum += wgt;
    const uint4 raw = *reinterpret_cast<const uint4*>(o_part + (s * rows + grow) * D + c8);
    const __bf16* h = reinterpret_cast<const __bf16*>(&raw);
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] += wgt * (float)h[j];
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
  // butterfly merge of (m, l, o) across the wave
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const float m2 = __shfl_xor(m, off), l2 = __shfl_xor(l, off);
    const float mn = fmaxf(m, m2);
    const float a1 = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - mn);
    const float a2 = m2 == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m2 - mn);
    l = l * a1 + l2 * a2;
#pragma unroll
    for (int e = 0; e < D; ++e) o[e] = o[e] * a1 + __shfl_xor(o[e], off) * a2;
    m = mn;
  }
  const float inv = 1.f / l;
  float* dst = a.out + rid * D;
  // every lane holds the merged row; lane e writes element e
#pragma unroll
  for (int e = 0; e < D; ++e)
    if (e % 64 == lane) dst[e] = o[e] * inv;
}

}  // namespace

AttnPlan make_attn_plan(const ckv_dims* d, int64_t k) {
  AttnPlan p{};
  const int G = d->n_q_heads / d->n_kv_heads;
  p.rows = G * d->n_suffix;
  if (d->dtype == CKV_DTYPE_F32) {  // one wave per row, no splits
    p.n_splits = 1;
    return p;
  }
  const int64_t np = k * d->chunk_size + d->n_suffix;
  const int64_t ntiles = ceil_div(np, kTile);
  const int64_t base = (int64_t)d->n_kv_heads * ceil_div(p.rows, kBlockRows);
  // at most ~2 workgroups per CU, keeping >= 4 stages per split; then the
  // fewest splits that give the same stages per split
  int64_t splits = std::max<int64_t>(1, 512 / base);
  splits = std::min<int64_t>(splits, std::max<int64_t>(1, ntiles / 4));
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
  a.q = static_cast<const uint16_t*>(q);
  a.kbase = static_cast<const uint16_t*>(src.k_base);
  a.vbase = static_cast<const uint16_t*>(src.v_base);
  a.chunk_stride = src.chunk_stride;
  a.chunk_off = src.chunk_off;
  a.direct = src.direct;
  a.sel = sel;
  a.kc = (int)(k * d->chunk_size);
  a.n = d->n_prefix;
  a.c = d->chunk_size;
  a.log2c = (d->chunk_size & (d->chunk_size - 1)) == 0 ? __builtin_ctz(d->chunk_size) : -1;
  a.short_tail = d->n_prefix % d->chunk_size ? (int)(d->chunk_size - d->n_prefix % d->chunk_size) : 0;
  a.ks = static_cast<const uint16_t*>(k_suffix);
  a.vs = static_cast<const uint16_t*>(v_suffix);
  a.out = static_cast<uint16_t*>(out);
  a.o_part = p.n_splits > 1 ? reinterpret_cast<uint16_t*>(static_cast<char*>(ws) + p.off_o) : nullptr;
  a.ml_part = p.n_splits > 1 ? reinterpret_cast<float2*>(static_cast<char*>(ws) + p.off_ml) : nullptr;
  a.S = d->n_suffix; a.Hq = d->n_q_heads; a.Hkv = d->n_kv_heads;
  a.G = d->n_q_heads / d->n_kv_heads; a.R = p.rows;
  a.n_splits = p.n_splits;
  const int64_t ntiles = ceil_div(a.kc + a.S, kTile);
  a.tiles_per_split = (int)ceil_div(ntiles, p.n_splits);
  a.n_row_blocks = (int)ceil_div(p.rows, kBlockRows);
  a.c1 = resolve_scale(d) * 1.4426950408889634f;
  a.nblocks = (uint32_t)((int64_t)a.Hkv * a.n_row_blocks * a.n_splits);
  a.nblocks_padded = (uint32_t)align_up(a.nblocks, 8);
  if (d->head_dim == 128)
    hipLaunchKernelGGL(attn_kernel<128>, dim3(a.nblocks_padded), dim3(kWaves * 64), 0, st, a);
  else
    hipLaunchKernelGGL(attn_kernel<64>, dim3(a.nblocks_padded), dim3(kWaves * 64), 0, st, a);
  CKV_HIP(hipGetLastError());
  if (p.n_splits > 1) {
    const int64_t work = (int64_t)a.Hkv * a.R * (d->head_dim / 8);
    if (d->head_dim == 128)
      hipLaunchKernelGGL(combine_kernel<128>, dim3((unsigned)ceil_div(work, 256)), dim3(256), 0, st,
                         a.o_part, a.ml_part, a.out, a.n_splits, a.Hkv, a.R, a.G, a.Hq);
    else
      hipLaunchKernelGGL(combine_kernel<64>, dim3((unsigned)ceil_div(work, 256)), dim3(256), 0, st,
                         a.o_part, a.ml_part, a.out, a.n_splits, a.Hkv, a.R, a.G, a.Hq);
    CKV_HIP(hipGetLastError());
  }
  return CKV_OK;
}

}  // namespace ckv
