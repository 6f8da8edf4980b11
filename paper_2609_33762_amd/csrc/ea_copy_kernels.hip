// Paged KV piece copies between the GPU cache and a slot-layout buffer.
//
// A "piece" is the contiguous K+V data of one (layer, page): 2*T*H*D*s
// bytes (8-64 KiB for the shapes this library serves).  One workgroup of
// 256 lanes (four wave64s) copies one piece per iteration of a grid-stride
// loop: every lane issues VEC independent 16-byte loads, then VEC stores, so
// each wave moves VEC contiguous KiB per round trip and a CU keeps
// 8 workgroups * 256 lanes * VEC * 16 B in flight, which is what HBM3E
// (and, for the direct host plans, the PCIe link's latency) needs.  The same
// kernel serves four transfers, differing only in where the slot-layout
// buffer lives and in the direction:
//   store  (cache -> mapped pinned host slots), load  (host slots -> cache),
//   gather (cache -> HBM staging),               scatter (HBM staging -> cache).
// Bytes are copied as opaque 16-byte vectors: fp8/bf16 payloads, NaN
// encodings included, are never interpreted.
#include <hip/hip_runtime.h>

#include "ea_internal.hpp"

namespace ea {
namespace {

constexpr int kThreads = 256;

template <int DIR, bool INLINE, int VEC>
__global__ __launch_bounds__(kThreads) void piece_copy_kernel(PieceCopy a,
                                                              InlineIdx inl) {
  const int64_t units = a.n * a.layer_count;
  const int64_t nvec = a.piece_bytes >> 4;
  const int tid = threadIdx.x;
  for (int64_t u = blockIdx.x; u < units; u += gridDim.x) {
    const int64_t i = u / a.layer_count;
    const int64_t l = a.layer_begin + (u - i * a.layer_count);
    int64_t page, slot;
    if constexpr (INLINE) {
      page = inl.pages[i];
      slot = inl.slots[i];
    } else {
      page = a.pages[i];
      slot = a.identity_slots ? i : a.slot_idx[i];
    }
    uint8_t *cache_piece = a.cache + (l * a.num_pages + page) * a.piece_bytes;
    uint8_t *slot_base = a.slots + slot * a.slot_bytes;
    uint8_t *slot_piece = slot_base + l * a.piece_bytes;
    const uint4 *src =
        reinterpret_cast<const uint4 *>(DIR == kToSlots ? cache_piece : slot_piece);
    uint4 *dst = reinterpret_cast<uint4 *>(DIR == kToSlots ? slot_piece : cache_piece);
    for (int64_t base = 0; base < nvec; base += (int64_t)kThreads * VEC) {
      uint4 r[VEC];
#pragma unroll
      for (int k = 0; k < VEC; ++k) {
        const int64_t v = base + k * kThreads + tid;
        if (v < nvec) r[k] = src[v];
      }
#pragma unroll
      for (int k = 0; k < VEC; ++k) {
        const int64_t v = base + k * kThreads + tid;
        if (v < nvec) dst[v] = r[k];
      }
    }
    if (a.scales != nullptr) {
      // 8 bytes (K scale, V scale) per (layer, page).  In a slot they sit in
      // the trailer after the page data, 8 bytes per layer, followed by zero
      // padding up to slot_bytes that a store writes with layer 0.
      uint64_t *cs = reinterpret_cast<uint64_t *>(a.scales + (l * a.num_pages + page) * 8);
      uint64_t *ss = reinterpret_cast<uint64_t *>(slot_base + a.page_bytes + l * 8);
      if (tid == 0) {
        if (DIR == kToSlots) *ss = *cs; else *cs = *ss;
      }
      if (DIR == kToSlots && l == 0) {
        const int64_t pad_begin = a.page_bytes + 8 * (int64_t)a.num_layers;
        const int64_t pad_words = (a.slot_bytes - pad_begin) >> 3;
        uint64_t *pad = reinterpret_cast<uint64_t *>(slot_base + pad_begin);
        for (int64_t w = tid; w < pad_words; w += kThreads) pad[w] = 0;
      }
    }
  }
}

template <int DIR, bool INLINE>
hipError_t launch_vec(const PieceCopy &a, const InlineIdx &inl, int64_t grid,
                      hipStream_t stream) {
  const int64_t nvec = a.piece_bytes >> 4;
  // enough vectors per lane to cover the piece in one pass, at most 8
  dim3 g((unsigned)grid), b(kThreads);
  if (nvec >= 8 * kThreads)
    hipLaunchKernelGGL((piece_copy_kernel<DIR, INLINE, 8>), g, b, 0, stream, a, inl);
  else if (nvec >= 4 * kThreads)
    hipLaunchKernelGGL((piece_copy_kernel<DIR, INLINE, 4>), g, b, 0, stream, a, inl);
  else if (nvec >= 2 * kThreads)
    hipLaunchKernelGGL((piece_copy_kernel<DIR, INLINE, 2>), g, b, 0, stream, a, inl);
  else
    hipLaunchKernelGGL((piece_copy_kernel<DIR, INLINE, 1>), g, b, 0, stream, a, inl);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_piece_copy(const PieceCopy &a, const InlineIdx *inl, int dir,
                             int grid_cap, hipStream_t stream) {
  const int64_t units = a.n * a.layer_count;
  if (units <= 0) return hipSuccess;
  // 256 CUs x 8 resident workgroups of 256 lanes fill the chip once; the
  // grid-stride loop covers the rest.
  int64_t cap = grid_cap > 0 ? grid_cap : 2048;
  int64_t grid = units < cap ? units : cap;
  static const InlineIdx kEmpty{};
  if (inl != nullptr) {
    return dir == kToSlots ? launch_vec<kToSlots, true>(a, *inl, grid, stream)
                           : launch_vec<kToPages, true>(a, *inl, grid, stream);
  }
  return dir == kToSlots ? launch_vec<kToSlots, false>(a, kEmpty, grid, stream)
                         : launch_vec<kToPages, false>(a, kEmpty, grid, stream);
}

}  // namespace ea
