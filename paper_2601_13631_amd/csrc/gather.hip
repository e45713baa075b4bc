// gather.hip -- contiguous ContiguousChunk gather (Sec. 4.2) for gfx950.
//
// Copies the K and V spans of the selected chunks into compact buffers, whole
// spans with 16-byte loads and stores, so exactly the selected bytes move (no
// block read amplification).  Rows past n of a short last chunk are zeroed.
// The source may be device memory or pinned host memory mapped into the device
// address space (then the loads cross the host link).
//
// Grid: x = 16-byte pieces of one chunk span (4 per thread), y = chunk, z = K/V.

#include "tiers_internal.h"

namespace ckv {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

__global__ __launch_bounds__(kThreads) void gather_kernel(const uint8_t* __restrict__ k_src,
                                                          const uint8_t* __restrict__ v_src,
                                                          const int32_t* __restrict__ sel,
                                                          uint8_t* __restrict__ k_dst,
                                                          uint8_t* __restrict__ v_dst, int64_t n,
                                                          int c, int64_t m, int64_t row_bytes) {
  const int64_t u = blockIdx.y;
  const uint8_t* src = blockIdx.z ? v_src : k_src;
  uint8_t* dst = blockIdx.z ? v_dst : k_dst;
  const int64_t slot_bytes = (int64_t)c * row_bytes;
  const int64_t j = sel[u];
  const bool ok = j >= 0 && j < m;
  const int64_t first = ok ? j * c : 0;
  const int64_t valid = ok ? min<int64_t>(c, n - first) * row_bytes : 0;
  const uint8_t* s = src + first * row_bytes;
  uint8_t* d = dst + u * slot_bytes;
  const int64_t base = ((int64_t)blockIdx.x * kThreads * kUnroll + threadIdx.x) * 16;
  // every load unconditional, at an offset clamped into the valid bytes (a
  // load behind its own predicate would wait for the one before it); pieces
  // past the valid bytes are zeroed afterwards
  const int64_t last = valid > 0 ? valid - 16 : 0;
  u32x4 v[kUnroll];
#pragma unroll
  for (int p = 0; p < kUnroll; ++p) {
    const int64_t off = base + (int64_t)p * kThreads * 16;
    v[p] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(s + min(off, last)));
  }
#pragma unroll
  for (int p = 0; p < kUnroll; ++p) {
    const int64_t off = base + (int64_t)p * kThreads * 16;
    if (off >= valid) v[p] = u32x4{0u, 0u, 0u, 0u};
    if (off < slot_bytes) *reinterpret_cast<u32x4*>(d + off) = v[p];
  }
}

// Whole-span copies for the host-resident prefix.  A small fixed grid walks
// all 16 KiB pieces of all listed spans (grid-stride), so the copy keeps
// thousands of 16-byte loads in flight over the host link -- one launch per
// list instead of one DMA copy per run of chunks -- while occupying only a
// few wave slots, next to the compute kernels it overlaps: 8 workgroups with
// every thread's four loads in flight at once (32 with one load at a time, or
// 16 with four, measured slower on the host-resident 128K-token layer).
constexpr int kCopyBlocks = 8;
// HBM-to-HBM slot moves (cache fills) run on the compute stream: a wider grid
constexpr int kSlotCopyBlocks = 256;

// dst_slots == nullptr: span i goes to slot slot0 + i.  span_bytes is a
// positive multiple of 16 (checked by the launchers).
__global__ __launch_bounds__(kThreads) void copy_spans_kernel(const uint8_t* __restrict__ src,
                                                              const int32_t* __restrict__ chunks,
                                                              int64_t count, int64_t slot0,
                                                              const int32_t* __restrict__ dst_slots,
                                                              uint8_t* __restrict__ dst,
                                                              int64_t span_bytes) {
  constexpr int64_t kPiece = (int64_t)kThreads * kUnroll * 16;
  const int64_t per_span = (span_bytes + kPiece - 1) / kPiece;
  const int64_t total = count * per_span;
  for (int64_t w = blockIdx.x; w < total; w += gridDim.x) {
    const int64_t i = w / per_span, piece = w % per_span;
    const uint8_t* s = src + (int64_t)chunks[i] * span_bytes;
    uint8_t* d = dst + (dst_slots ? (int64_t)dst_slots[i] : slot0 + i) * span_bytes;
    const int64_t base = piece * kPiece + (int64_t)threadIdx.x * 16;
    // unconditional loads at offsets clamped into the span (see gather_kernel)
    u32x4 v[kUnroll];
#pragma unroll
    for (int p = 0; p < kUnroll; ++p) {
      const int64_t off = base + (int64_t)p * kThreads * 16;
      v[p] = __builtin_nontemporal_load(
          reinterpret_cast<const u32x4*>(s + min(off, span_bytes - 16)));
    }
#pragma unroll
    for (int p = 0; p < kUnroll; ++p) {
      const int64_t off = base + (int64_t)p * kThreads * 16;
      if (off < span_bytes) *reinterpret_cast<u32x4*>(d + off) = v[p];
    }
  }
}

}  // namespace

ckv_status launch_copy_spans(const void* src, const int32_t* chunks, int64_t count, int64_t slot0,
                             void* dst, int64_t span_bytes, hipStream_t st) {
  if (span_bytes <= 0 || span_bytes % 16 != 0)
    CKV_FAIL(CKV_EINVAL, "span bytes must be a positive multiple of 16");
  if (count == 0) return CKV_OK;
  const int64_t pieces = count * ceil_div(span_bytes, (int64_t)kThreads * kUnroll * 16);
  const unsigned grid = (unsigned)std::min<int64_t>(pieces, kCopyBlocks);
  hipLaunchKernelGGL(copy_spans_kernel, dim3(grid), dim3(kThreads), 0, st,
                     static_cast<const uint8_t*>(src), chunks, count, slot0, nullptr,
                     static_cast<uint8_t*>(dst), span_bytes);
  CKV_HIP(hipGetLastError());
  return CKV_OK;
}

ckv_status launch_copy_slots(const void* src, const int32_t* src_slots, void* dst,
                             const int32_t* dst_slots, int64_t count, int64_t span_bytes,
                             hipStream_t st) {
  if (span_bytes <= 0 || span_bytes % 16 != 0)
    CKV_FAIL(CKV_EINVAL, "span bytes must be a positive multiple of 16");
  if (count == 0) return CKV_OK;
  const int64_t pieces = count * ceil_div(span_bytes, (int64_t)kThreads * kUnroll * 16);
  const unsigned grid = (unsigned)std::min<int64_t>(pieces, kSlotCopyBlocks);
  hipLaunchKernelGGL(copy_spans_kernel, dim3(grid), dim3(kThreads), 0, st,
                     static_cast<const uint8_t*>(src), src_slots, count, 0, dst_slots,
                     static_cast<uint8_t*>(dst), span_bytes);
  CKV_HIP(hipGetLastError());
  return CKV_OK;
}

const void* device_view(const void* p) {
  hipPointerAttribute_t at{};
  if (hipPointerGetAttributes(&at, p) != hipSuccess) {
    (void)hipGetLastError();  // pageable memory: clear the error the query left
    return nullptr;
  }
  if (at.type == hipMemoryTypeDevice || at.type == hipMemoryTypeManaged ||
      at.type == hipMemoryTypeUnified)
    return p;
  if (at.type == hipMemoryTypeHost) {
    if (!at.devicePointer) return p;
    // the device address of p itself, whether the query reported p or the
    // start of its allocation
    const char* hp = static_cast<const char*>(at.hostPointer ? at.hostPointer : p);
    return static_cast<const char*>(at.devicePointer) + (static_cast<const char*>(p) - hp);
  }
  return nullptr;
}

ckv_status launch_gather(const ckv_dims* d, const void* k_src, const void* v_src,
                         const int32_t* sel, int64_t k, void* k_dst, void* v_dst, hipStream_t st) {
  if (k == 0) return CKV_OK;
  const int64_t row_bytes = (int64_t)d->n_kv_heads * d->head_dim * elem_bytes(d->dtype);
  const int64_t slot_bytes = row_bytes * d->chunk_size;
  const int64_t m = ceil_div(d->n_prefix, d->chunk_size);
  dim3 grid((unsigned)ceil_div(slot_bytes, (int64_t)kThreads * kUnroll * 16), (unsigned)k, 2);
  hipLaunchKernelGGL(gather_kernel, grid, dim3(kThreads), 0, st,
                     static_cast<const uint8_t*>(k_src), static_cast<const uint8_t*>(v_src), sel,
                     static_cast<uint8_t*>(k_dst), static_cast<uint8_t*>(v_dst), d->n_prefix,
                     d->chunk_size, m, row_bytes);
  CKV_HIP(hipGetLastError());
  return CKV_OK;
}

}  // namespace ckv
