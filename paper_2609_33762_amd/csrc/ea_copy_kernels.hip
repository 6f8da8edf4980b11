// Paged KV piece copies between the GPU cache and a slot-layout buffer.
//
// A "piece" is the contiguous K+V data of one (layer, page): 2*T*H*D*s
// bytes (8-64 KiB for the shapes this library serves).  Each wave64 copies
// whole pieces on its own (grid-stride over (entry, layer) units): per round
// every lane issues VEC independent 16-byte non-temporal loads and then the
// VEC stores, so a wave moves VEC contiguous KiB per round trip and needs no
// barrier or LDS.  Non-temporal accesses stream past L2 and the MALL (the
// data is touched once).  The same kernel serves four transfers, differing
// only in where the slot-layout buffer lives and in the direction:
//   store  (cache -> mapped pinned host slots), load  (host slots -> cache),
//   gather (cache -> HBM staging),               scatter (HBM staging -> cache).
// Bytes move as opaque 16-byte vectors: fp8/bf16 payloads, NaN encodings
// included, are never interpreted.
//
// The per-vector bounds checks make the compiler let each store wait for
// the one before it.  On MI355X that measured faster than a loop without
// the checks that keeps all stores of a round in flight: the paged gather
// reached 5.66 TB/s against 5.28-5.37, and a store and a load sharing the
// PCIe link reached 79.6 GB/s together against 72.9 (fewer posted writes in
// flight leave room for the load's read requests).
#include <hip/hip_runtime.h>

#include "ea_internal.hpp"

namespace ea {
namespace {

constexpr int kThreads = 256;  // four wave64s per workgroup
constexpr int kWave = 64;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// s_getreg operand for HW_REG_XCC_ID (hardware register 20), bits [3:0]:
// the XCD the wave runs on.
constexpr int kXccIdReg = (3 << 11) | (0 << 6) | 20;

__device__ __forceinline__ int this_xcd(const PieceCopy &a) {
  if (a.hw_xcd) return (int)((__builtin_amdgcn_s_getreg(kXccIdReg) & 0xFu) % (unsigned)a.num_xcd);
  return (int)(blockIdx.x % (unsigned)a.num_xcd);
}

__device__ __forceinline__ u32x4 load_nt(const u32x4 *p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void store_nt(u32x4 *p, u32x4 v) { __builtin_nontemporal_store(v, p); }

// Unit u is (entry i, layer l): entry-major (u = i * layer_count + l - b,
// a page's layers one after the other) or, with a.layer_major, layer-major
// (u = (l - b) * n + i, every entry of one layer first); b = layer_begin.
__device__ __forceinline__ int64_t unit_entry(const PieceCopy &a, int64_t u) {
  return a.layer_major ? u % a.n : u / a.layer_count;
}
__device__ __forceinline__ int64_t unit_layer(const PieceCopy &a, int64_t u, int64_t i) {
  return a.layer_begin + (a.layer_major ? u / a.n : u - i * a.layer_count);
}

// Copy the piece of layer l of entry i, whose page and slot the caller has
// made wave-uniform.  The entry's piece sits at chunk position c = i mod C
// of layer l inside the slot.
template <int DIR, bool INLINE, int VEC>
__device__ __forceinline__ void copy_unit(const PieceCopy &a, int64_t l, int64_t i, int64_t page,
                                          int64_t slot, int lane) {
  const int64_t nvec = a.piece_bytes >> 4;
  const int64_t c = a.chunk == 1 ? 0 : (int64_t)((uint32_t)i % (uint32_t)a.chunk);
  const int64_t at = l * a.chunk + c;  // piece index inside the slot
  uint8_t *cache_piece = a.cache + (l * a.num_pages + page) * a.piece_bytes;
  uint8_t *slot_base = a.slots + slot * a.slot_bytes;
  uint8_t *slot_piece = slot_base + at * a.piece_bytes;
  const u32x4 *src = reinterpret_cast<const u32x4 *>(DIR == kToSlots ? cache_piece : slot_piece);
  u32x4 *dst = reinterpret_cast<u32x4 *>(DIR == kToSlots ? slot_piece : cache_piece);
  // The scale word is read before the piece, so that its round trip (over
  // the host link for a load) overlaps the piece's instead of following it.
  uint64_t *cs = nullptr, *ss = nullptr;
  uint64_t scale = 0;
  if (a.scales != nullptr) {
    cs = reinterpret_cast<uint64_t *>(a.scales + (l * a.num_pages + page) * 8);
    ss = reinterpret_cast<uint64_t *>(slot_base + a.payload_bytes + at * 8);
    if (lane == 0) scale = DIR == kToSlots ? *cs : *ss;
  }
  for (int64_t base = 0; base < nvec; base += (int64_t)kWave * VEC) {
    u32x4 r[VEC];
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
      const int64_t v = base + k * kWave + lane;
      if (v < nvec) r[k] = load_nt(src + v);
    }
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
      const int64_t v = base + k * kWave + lane;
      if (v < nvec) store_nt(dst + v, r[k]);
    }
  }
  if (a.scales != nullptr) {
    if (lane == 0) {
      if (DIR == kToSlots) *ss = scale; else *cs = scale;
    }
    if (DIR == kToSlots && at == 0) {  // once per slot
      const int64_t pad_begin = a.payload_bytes + 8 * (int64_t)a.num_layers * a.chunk;
      const int64_t pad_words = (a.slot_bytes - pad_begin) >> 3;
      uint64_t *pad = reinterpret_cast<uint64_t *>(slot_base + pad_begin);
      for (int64_t w = lane; w < pad_words; w += kWave) pad[w] = 0;
    }
  }
}

// Loads first on the host link.  Every wave of a load raises the tier's
// counter for its whole loop.  A store wave reads the counter before each
// unit and acts on it after the unit (so the read's round trip overlaps the
// copy): while a load runs it sleeps a.yield_units x 1,024 cycles per 32 KiB
// copied, which holds back small pieces as much as large ones.
constexpr int64_t kYieldBytes = 32768;

__device__ __forceinline__ uint32_t link_busy(const PieceCopy &a) {
  if (a.link_role != kLinkYield) return 0;
  return __hip_atomic_load(a.link_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void yield_link(const PieceCopy &a, uint32_t busy, int64_t &debt) {
  if (a.link_role != kLinkYield) return;
  debt += a.piece_bytes;
  if (__builtin_amdgcn_readfirstlane(busy) == 0) {
    debt = 0;  // nothing to make up once the link is free
    return;
  }
  for (; debt >= kYieldBytes; debt -= kYieldBytes)
    for (int32_t k = 0; k < a.yield_units; ++k) __builtin_amdgcn_s_sleep(16);  // 16 x 64 cycles
}
// one lane per wave: +1 before a load wave's loop, -1 after it
__device__ __forceinline__ void mark_load(const PieceCopy &a, int lane, int32_t delta) {
  if (a.link_role == kLinkMark && lane == 0)
    __hip_atomic_fetch_add(a.link_flag, (uint32_t)delta, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

template <int DIR, bool INLINE, int VEC>
__device__ __forceinline__ void piece_copy(const PieceCopy &a, const int32_t *__restrict__ pages,
                                           const int64_t *__restrict__ slot_idx,
                                           const InlineIdx *inl) {
  const int64_t units = a.n * a.layer_count;
  const int lane = threadIdx.x & (kWave - 1);
  const int xcd = this_xcd(a);
  if (!((a.xcd_mask >> xcd) & 1u)) return;
  const int active = __popc(a.xcd_mask);
  const int64_t group = (int64_t)(blockIdx.x / (unsigned)a.num_xcd) * active +
                        __popc(a.xcd_mask & ((1u << xcd) - 1u));
  const int64_t groups = (int64_t)(gridDim.x / (unsigned)a.num_xcd) * active;
  const int64_t waves = groups * (kThreads / kWave);
  const int64_t first =
      group * (kThreads / kWave) + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  int64_t debt = 0;  // bytes a yielding store has copied since its last sleep
  mark_load(a, lane, 1);
  if constexpr (INLINE) {
    // indices from the kernel arguments (scalar loads, u is wave-uniform)
    for (int64_t u = first; u < units; u += waves) {
      const int64_t i = unit_entry(a, u);
      const uint32_t busy = link_busy(a);
      copy_unit<DIR, INLINE, VEC>(a, unit_layer(a, u, i), i, inl->pages[i], inl->slots[i], lane);
      yield_link(a, busy, debt);
    }
  } else {
    // The index arrays live in pinned host memory that the kernel reads
    // over the link, or in the kernel arguments.  Lane k fetches the page
    // and slot of the wave's k-th next unit in one vector load per 64
    // units, and the loop broadcasts them with readlane, so a unit's copy
    // never waits on an index fetch.
    for (int64_t k0 = 0;; k0 += kWave) {
      const int64_t u0 = first + k0 * waves;
      if (u0 >= units) break;
      const int64_t ul = u0 + (int64_t)lane * waves;
      int32_t vpage = 0;
      int64_t vslot = 0;
      if (ul < units) {
        const int64_t il = unit_entry(a, ul);
        vpage = pages[il];
        vslot = a.identity_slots ? (int64_t)((uint32_t)il / (uint32_t)a.chunk) : slot_idx[il];
      }
      for (int k = 0; k < kWave; ++k) {
        const int64_t u = u0 + (int64_t)k * waves;
        if (u >= units) break;
        const int64_t i = unit_entry(a, u);
        const int64_t page = __builtin_amdgcn_readlane(vpage, k);
        const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)vslot, k);
        const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)vslot >> 32), k);
        const uint32_t busy = link_busy(a);
        copy_unit<DIR, INLINE, VEC>(a, unit_layer(a, u, i), i, page,
                                    (int64_t)(((uint64_t)hi << 32) | lo), lane);
        yield_link(a, busy, debt);
      }
    }
  }
  mark_load(a, lane, -1);
}

// Two entry points with the same body, so that profiles tell the host-link
// transfers (direct store/load, few workgroups) from the HBM gather/scatter.
template <int DIR, bool INLINE, int VEC>
__global__ __launch_bounds__(kThreads) void copy_host_link(PieceCopy a,
                                                           const int32_t *__restrict__ pages,
                                                           const int64_t *__restrict__ slot_idx,
                                                           InlineIdx inl) {
  piece_copy<DIR, INLINE, VEC>(a, pages, slot_idx, &inl);
}
template <int DIR, bool INLINE, int VEC>
__global__ __launch_bounds__(kThreads) void copy_hbm(PieceCopy a, const int32_t *__restrict__ pages,
                                                     const int64_t *__restrict__ slot_idx,
                                                     InlineIdx inl) {
  piece_copy<DIR, INLINE, VEC>(a, pages, slot_idx, &inl);
}
// The HBM gather/scatter with the page ids of up to kArgPagesMax entries in
// the kernel arguments (slot of entry i is i): the same loop reads them as
// it reads an index array, and the call needs no index buffer whose reuse
// the host would have to track.
template <int DIR, int VEC>
__global__ __launch_bounds__(kThreads) void copy_hbm_args(PieceCopy a, ArgPages ids) {
  piece_copy<DIR, false, VEC>(a, ids.pages, nullptr, nullptr);
}

// Consumer stand-in of the layered load: wave w of the grid folds the
// pieces of pages w, w + waves, ... of one layer into the XOR of their
// little-endian 64-bit words (and the page's scale word), one 16-byte
// vector per lane per step, then across the wave by lane swaps.
__global__ __launch_bounds__(kThreads) void layer_checksum(
    const uint8_t *__restrict__ cache, const uint8_t *__restrict__ scales, int64_t num_pages,
    int64_t piece_bytes, int32_t layer, const int32_t *__restrict__ pages, int32_t n,
    uint64_t *__restrict__ out) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t waves = (int64_t)gridDim.x * (kThreads / kWave);
  const int64_t first = (int64_t)blockIdx.x * (kThreads / kWave) +
                        __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int64_t nvec = piece_bytes >> 4;
  for (int64_t i = first; i < n; i += waves) {
    const int64_t page = pages[i];
    const u32x4 *src =
        reinterpret_cast<const u32x4 *>(cache + ((int64_t)layer * num_pages + page) * piece_bytes);
    uint32_t lo = 0, hi = 0;
    for (int64_t v = lane; v < nvec; v += kWave) {
      const u32x4 x = src[v];
      lo ^= x.x ^ x.z;
      hi ^= x.y ^ x.w;
    }
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
      lo ^= (uint32_t)__shfl_xor((int)lo, d, kWave);
      hi ^= (uint32_t)__shfl_xor((int)hi, d, kWave);
    }
    if (lane == 0) {
      uint64_t x = ((uint64_t)hi << 32) | lo;
      if (scales != nullptr)
        x ^= *reinterpret_cast<const uint64_t *>(scales + ((int64_t)layer * num_pages + page) * 8);
      out[i] = x;
    }
  }
}

// One workgroup of one wave per entry: out[b] = the XCD of workgroup b.
__global__ __launch_bounds__(64) void xcd_probe(int32_t *__restrict__ out) {
  if (threadIdx.x == 0) out[blockIdx.x] = (int32_t)(__builtin_amdgcn_s_getreg(kXccIdReg) & 0xFu);
}

template <int DIR, bool INLINE, int VEC>
void launch_route(const PieceCopy &a, const InlineIdx &inl, const ArgPages *ids, int route, dim3 g,
                  hipStream_t stream) {
  if (ids != nullptr)
    hipLaunchKernelGGL((copy_hbm_args<DIR, VEC>), g, dim3(kThreads), 0, stream, a, *ids);
  else if (route == kRouteHostLink)
    hipLaunchKernelGGL((copy_host_link<DIR, INLINE, VEC>), g, dim3(kThreads), 0, stream, a,
                       a.pages, a.slot_idx, inl);
  else
    hipLaunchKernelGGL((copy_hbm<DIR, INLINE, VEC>), g, dim3(kThreads), 0, stream, a, a.pages,
                       a.slot_idx, inl);
}

template <int DIR, bool INLINE>
void launch_dir(const PieceCopy &a, const InlineIdx &inl, const ArgPages *ids, int route,
                int64_t grid, hipStream_t stream) {
  const dim3 g((unsigned)grid);
  const int64_t nvec = a.piece_bytes >> 4;
  // four vectors per lane per round measured best for 8-64 KiB pieces; a
  // piece smaller than one round uses fewer
  if (nvec >= 4 * kWave) launch_route<DIR, INLINE, 4>(a, inl, ids, route, g, stream);
  else if (nvec >= 2 * kWave) launch_route<DIR, INLINE, 2>(a, inl, ids, route, g, stream);
  else launch_route<DIR, INLINE, 1>(a, inl, ids, route, g, stream);
}

}  // namespace

hipError_t probe_xcd_round_robin(int num_xcd, bool *ok) {
  *ok = false;
  if (num_xcd < 1 || num_xcd > 16) return hipSuccess;
  const int most = 8 * num_xcd;
  // a private stream: the probe stays off the legacy default stream
  hipStream_t s = nullptr;
  hipError_t e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
  if (e != hipSuccess) return e;
  int32_t *d = nullptr;
  if ((e = hipMalloc((void **)&d, (size_t)most * sizeof(int32_t))) != hipSuccess) {
    (void)hipStreamDestroy(s);
    return e;
  }
  int32_t h[128];
  bool good = true;
  // several dispatch sizes, each twice: the offset may change between
  // dispatches, the round-robin order within one must not
  for (int rep = 0; rep < 2 && good && e == hipSuccess; ++rep) {
    for (int grid : {num_xcd, 3 * num_xcd, 8 * num_xcd}) {
      (void)hipGetLastError();
      hipLaunchKernelGGL(xcd_probe, dim3((unsigned)grid), dim3(64), 0, s, d);
      if ((e = hipGetLastError()) != hipSuccess) break;
      if ((e = hipMemcpyAsync(h, d, (size_t)grid * sizeof(int32_t), hipMemcpyDeviceToHost, s)) !=
          hipSuccess)
        break;
      if ((e = hipStreamSynchronize(s)) != hipSuccess) break;
      for (int b = 0; b < grid && good; ++b)
        good = h[b] >= 0 && h[b] % num_xcd == (h[0] % num_xcd + b) % num_xcd;
      if (!good) break;
    }
  }
  (void)hipStreamSynchronize(s);
  (void)hipFree(d);
  (void)hipStreamDestroy(s);
  if (e == hipSuccess) *ok = good;
  return e;
}

hipError_t launch_layer_checksum(const uint8_t *cache, const uint8_t *scales, int64_t num_pages,
                                 int64_t piece_bytes, int32_t layer, const int32_t *pages,
                                 int32_t n, uint64_t *out, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int64_t waves_per_group = kThreads / kWave;
  int64_t grid = (n + waves_per_group - 1) / waves_per_group;
  if (grid > 1024) grid = 1024;
  (void)hipGetLastError();
  hipLaunchKernelGGL(layer_checksum, dim3((unsigned)grid), dim3(kThreads), 0, stream, cache,
                     scales, num_pages, piece_bytes, layer, pages, n, out);
  return hipGetLastError();
}

hipError_t launch_piece_copy(const PieceCopy &a, const InlineIdx *inl, const ArgPages *ids,
                             int dir, int route, int64_t workgroups, hipStream_t stream) {
  const int64_t units = a.n * a.layer_count;
  if (units <= 0) return hipSuccess;
  if (a.num_xcd < 1 || a.num_xcd > 32 || a.xcd_mask == 0 ||
      (a.num_xcd < 32 && (a.xcd_mask >> a.num_xcd) != 0))
    return hipErrorInvalidValue;
  // entry indices and chunk positions are computed in 32 bits
  if (a.chunk < 1 || a.n > INT32_MAX) return hipErrorInvalidValue;
  // page ids in the arguments: HBM route, identity slots, all ids there
  if (ids != nullptr && (inl != nullptr || route != kRouteHbm || !a.identity_slots ||
                         a.n > kArgPagesMax))
    return hipErrorInvalidValue;
  const int64_t waves_per_group = kThreads / kWave;
  const int64_t needed = (units + waves_per_group - 1) / waves_per_group;
  const int64_t work = needed < workgroups ? needed : workgroups;
  const int64_t active = __builtin_popcount(a.xcd_mask);
  // each run of num_xcd consecutive workgroups holds `active` working ones
  const int64_t grid = (work + active - 1) / active * a.num_xcd;
  static const InlineIdx kEmpty{};
  // report this launch's status only: drop any error an earlier runtime call
  // left recorded on this thread (hipGetLastError returns and clears it)
  (void)hipGetLastError();
  if (inl != nullptr) {
    if (dir == kToSlots) launch_dir<kToSlots, true>(a, *inl, nullptr, route, grid, stream);
    else launch_dir<kToPages, true>(a, *inl, nullptr, route, grid, stream);
  } else {
    if (dir == kToSlots) launch_dir<kToSlots, false>(a, kEmpty, ids, route, grid, stream);
    else launch_dir<kToPages, false>(a, kEmpty, ids, route, grid, stream);
  }
  return hipGetLastError();
}

}  // namespace ea
