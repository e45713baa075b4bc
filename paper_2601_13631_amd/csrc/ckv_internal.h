// ckv_internal.h -- internals shared by the libckv translation units (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <string>

#include "../../include/ckv.h"

namespace ckv {

// ---- error reporting -------------------------------------------------------
void set_error(const char* fmt, ...);
void clear_error();

#define CKV_FAIL(code, ...)   \
  do {                        \
    ::ckv::set_error(__VA_ARGS__); \
    return (code);            \
  } while (0)

#define CKV_HIP(call)                                                                   \
  do {                                                                                  \
    hipError_t e_ = (call);                                                             \
    if (e_ != hipSuccess)                                                               \
      CKV_FAIL(CKV_EHIP, "%s failed: %s (%d) at %s:%d", #call, hipGetErrorString(e_),   \
               (int)e_, __FILE__, __LINE__);                                            \
  } while (0)

// ---- vector types ----------------------------------------------------------
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) short s16x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

// ---- cross-lane moves without LDS ----------------------------------------------
// DPP inside a row of 16 lanes, and the gfx950 permlane swaps across rows.  A
// swap hands each lane its own value and its partner's (lane ^ 16 or ^ 32) in
// some order, which is all a symmetric reduction (min, max) needs.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, true);
}
constexpr int kDppQuadXor1 = 0xB1, kDppQuadXor2 = 0x4E, kDppRowHalfMirror = 0x141,
              kDppRowMirror = 0x140;
constexpr int kDppRowShr1 = 0x111, kDppRowShr2 = 0x112, kDppRowShr4 = 0x114, kDppRowShr8 = 0x118;

__device__ __forceinline__ uint64_t join64(uint32_t h, uint32_t l) { return ((uint64_t)h << 32) | l; }

template <int CTRL>
__device__ __forceinline__ uint64_t dpp64(uint64_t v) {
  return join64(dpp32<CTRL>((uint32_t)(v >> 32)), dpp32<CTRL>((uint32_t)v));
}

// (own, partner) of a 64-bit value for partner lane ^ 16 (WIDTH 16) or ^ 32.
template <int WIDTH>
__device__ __forceinline__ void swap_pair64(uint64_t v, uint64_t& a, uint64_t& b) {
  const uint32_t l = (uint32_t)v, h = (uint32_t)(v >> 32);
  if constexpr (WIDTH == 16) {
    const auto rl = __builtin_amdgcn_permlane16_swap(l, l, false, false);
    const auto rh = __builtin_amdgcn_permlane16_swap(h, h, false, false);
    a = join64(rh[0], rl[0]);
    b = join64(rh[1], rl[1]);
  } else {
    const auto rl = __builtin_amdgcn_permlane32_swap(l, l, false, false);
    const auto rh = __builtin_amdgcn_permlane32_swap(h, h, false, false);
    a = join64(rh[0], rl[0]);
    b = join64(rh[1], rl[1]);
  }
}

// ---- shape checks ------------------------------------------------------------
inline int elem_bytes(int dtype) { return dtype == CKV_DTYPE_F32 ? 4 : 2; }

// Validates the shape fields; returns CKV_OK, CKV_EINVAL or CKV_EUNSUPPORTED
// and records the reason.
ckv_status check_dims(const ckv_dims* d);

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline float resolve_scale(const ckv_dims* d) {
  return d->sm_scale > 0.f ? d->sm_scale : 1.0f / sqrtf((float)d->head_dim);
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// ---- launch helpers ------------------------------------------------------------
// Workgroups are dispatched round-robin over the 8 XCDs (blockIdx % 8).  This
// maps a hardware block id to a logical id so that consecutive logical ids run
// on the same XCD and share its L2.  nblocks_padded is a multiple of 8.
__device__ __forceinline__ uint32_t xcd_remap(uint32_t bid, uint32_t nblocks_padded) {
  return (bid & 7u) * (nblocks_padded >> 3) + (bid >> 3);
}

// ---- kernels' host-side launchers (each file owns its kernels) ----------------
// Work decomposition of chunk scoring.  Each (KV head g, row block rb) pair --
// rbh = g*RB + rb, a block of rpb rows of that head -- spans the whole key axis,
// cut into U units of UK keys (UK = lcm(64, c): whole 64-key stages and whole
// chunks).  The units of every rbh are split into NS segments of floor or ceil
// of U/NS units: segment s holds units [s*U/NS, (s+1)*U/NS).  One workgroup
// runs one segment, so the grid is Hkv*RB*NS workgroups of equal work (within
// one unit); NS is chosen so that the grid fills two workgroups per CU.
struct ScoreWork {
  int32_t rpb;  // rows per row block (a power of two)
  int32_t RB;   // row blocks per KV head
  int32_t UK;   // keys per unit
  int32_t U;    // units per rbh: ceil(n / UK)
  int32_t NS;   // segments per rbh
  int32_t ldp;  // row stride of the partial sums: RB * rpb
  __host__ __device__ int seg_begin(int s) const {  // first unit of segment s
    return (int)((int64_t)s * U / NS);
  }
  __host__ __device__ int seg_of_unit(int u) const {  // segment holding unit u
    return (int)((((int64_t)u + 1) * NS - 1) / U);
  }
};

struct ScorePlan {
  int64_t m;      // chunks
  int32_t rows;   // G*S rows per KV head
  ScoreWork w;
  // workspace layout: partial sums [Hkv][U*UK/c][ldp] (fp32), references
  // [Hkv*RB][NS][rpb] (fp32), sums / weights [Hkv*RB][NS][rpb] (fp64),
  // overflow flags [Hkv*RB][NS]
  size_t off_part, off_mc, off_z, off_flags, bytes;
};
ScorePlan make_score_plan(const ckv_dims* d);
// Optional timing of the main kernel: main_stop is recorded between the main
// kernel and the fold; main_span (bf16 only; score_span_words(d) words)
// receives every workgroup's start and end, in ticks of the 100 MHz realtime
// counter (the kernel's span is the earliest start to the latest end).
int64_t score_span_words(const ckv_dims* d);
ckv_status launch_score(const ckv_dims* d, const void* q, const void* k, double* scores,
                        void* ws, size_t ws_bytes, hipStream_t st,
                        hipEvent_t main_stop = nullptr, unsigned long long* main_span = nullptr);

size_t select_ws_bytes(int64_t m);
// sel_copy (optional, device): a second array that receives the same k indices.
ckv_status launch_select(const double* scores, int64_t m, int64_t k, int32_t* sel, void* ws,
                         size_t ws_bytes, hipStream_t st, int32_t* sel_copy = nullptr);

// Chunk addressing for gather/attention: chunk u's K rows start at
// k_base + off(u) * chunk_stride elements (V likewise from v_base), where
// off(u) = chunk_off ? chunk_off[u] : (direct ? sel[u] : u).  Row stride inside a
// chunk is Hkv*d elements.
struct ChunkSource {
  const void* k_base;
  const void* v_base;
  int64_t chunk_stride;     // elements between consecutive chunk slots
  const int32_t* chunk_off; // optional per-chunk slot table (device)
  int32_t direct;           // 1: off(u) = sel[u]; 0: off(u) = u (unless chunk_off)
  int64_t n_slots;          // slots the source holds (every off(u) is below it)
};

// Copies whole chunk spans of span_bytes each (16-byte multiple): span chunks[i]
// of src (pinned host memory mapped into the device address space, or device
// memory) to span slot0 + i of dst, for i < count; chunks is a device array.
ckv_status launch_copy_spans(const void* src, const int32_t* chunks, int64_t count, int64_t slot0,
                             void* dst, int64_t span_bytes, hipStream_t st);
// The address under which kernels read p: p itself for device memory, the
// mapped address for pinned host memory; nullptr if the device cannot read it
// (pageable host memory), which callers turn into CKV_EINVAL.
const void* device_view(const void* p);
ckv_status launch_gather(const ckv_dims* d, const void* k_src, const void* v_src,
                         const int32_t* sel, int64_t k, void* k_dst, void* v_dst, hipStream_t st);

struct AttnPlan {
  int32_t rows;      // G*S rows per KV head
  int32_t n_splits;  // key splits (1: no combine)
  size_t off_o, off_ml, bytes;
};
// Keys: the k kept chunks, then (with_suffix) the causal suffix.
AttnPlan make_attn_plan(const ckv_dims* d, int64_t k, bool with_suffix = true);
ckv_status launch_attn(const ckv_dims* d, const void* q, const ChunkSource& src,
                       const int32_t* sel, int64_t k, const void* k_suffix, const void* v_suffix,
                       void* out, void* ws, size_t ws_bytes, hipStream_t st);
// Attention in parts over one kept set (bf16): each part is a launch over
// some of the kept chunks (the first part with the suffix) that writes its
// split partials at split_base.. of a shared workspace, and one combine merges
// the n_splits partials of all parts in split order.  The parts may wait on
// different events: a host-resident layer attends over the chunks already in
// HBM while the rest (the late chunks) are still being copied, and over each
// share of the late chunks once its copy has landed.  The n_late late chunks
// go in parts = min(max_late_parts, n_late) consecutive non-empty shares,
// share i beginning at attn_late_part_begin(n_late, parts, i).
// attn_parted_splits is the most splits any division of k chunks into a
// first part and its late shares takes; attn_parted_bytes the workspace for
// that many.
int64_t attn_late_part_begin(int64_t n_late, int parts, int i);
int64_t attn_parted_splits(const ckv_dims* d, int64_t k, int max_late_parts);
size_t attn_parted_bytes(const ckv_dims* d, int64_t max_splits);
ckv_status launch_attn_part(const ckv_dims* d, const void* q, const ChunkSource& src,
                            const int32_t* sel, int64_t k, const void* k_suffix,
                            const void* v_suffix, bool with_suffix, void* ws, int64_t max_splits,
                            int32_t split_base, int32_t* n_splits, hipStream_t st);
ckv_status launch_attn_combine(const ckv_dims* d, const void* ws, int64_t max_splits,
                               int32_t n_splits, void* out, hipStream_t st);

}  // namespace ckv
