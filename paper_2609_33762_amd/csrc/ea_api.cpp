// C ABI of libea (include/ea.h): validation, pinned host tier, transfer
// plans, stream/event bookkeeping, gather/scatter and the peak probe.
#include <hip/hip_runtime_api.h>
#include <sys/syscall.h>
#include <unistd.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <memory>
#include <mutex>
#include <new>
#include <vector>

#include "ea.h"
#include "ea_internal.hpp"
#include "ea_tier_meta.hpp"

namespace {

thread_local int g_last_hip = 0;

#define EA_HIP(expr)          \
  do {                        \
    hipError_t e_ = (expr);   \
    if (e_ != hipSuccess) {   \
      g_last_hip = (int)e_;   \
      return EA_EHIP;         \
    }                         \
  } while (0)

#define EA_TRY(expr)              \
  do {                            \
    int rc_ = (expr);             \
    if (rc_ != EA_OK) return rc_; \
  } while (0)

// Make `dev` current for the duration of a call.
class DeviceScope {
 public:
  explicit DeviceScope(int dev) {
    if (hipGetDevice(&prev_) != hipSuccess) prev_ = -1;
    if (prev_ != dev) {
      err_ = hipSetDevice(dev);
      changed_ = err_ == hipSuccess;
    }
  }
  ~DeviceScope() {
    if (changed_ && prev_ >= 0) (void)hipSetDevice(prev_);
  }
  int status() const {
    if (err_ != hipSuccess) {
      g_last_hip = (int)err_;
      return EA_EHIP;
    }
    return EA_OK;
  }

 private:
  int prev_ = -1;
  bool changed_ = false;
  hipError_t err_ = hipSuccess;
};

int env_int(const char *name, int dflt) {
  const char *v = std::getenv(name);
  return v && *v ? std::atoi(v) : dflt;
}

// Pinned, device-mapped host memory.  The driver hands the pages of a
// buffer freed moments earlier back to its pool only some time later (on
// MI355X, 64 GiB freed by one tier became allocatable again 2.6 s after the
// free), so a tier created right after another was destroyed can fail for a
// while.  An out-of-memory failure is retried with growing waits for up to
// EA_HOST_ALLOC_WAIT_MS milliseconds (default 5000, 0 = no retry); a request
// larger than the machine's physical memory fails at once.
hipError_t host_alloc_retry(void **p, size_t bytes, unsigned flags) {
  hipError_t e = hipHostMalloc(p, bytes, flags);
  const long pages = sysconf(_SC_PHYS_PAGES), page = sysconf(_SC_PAGESIZE);
  if (e != hipErrorOutOfMemory || pages <= 0 || page <= 0 ||
      bytes > (size_t)pages * (size_t)page)
    return e;
  long budget_ms = std::max(0, env_int("EA_HOST_ALLOC_WAIT_MS", 5000));
  for (long wait_ms = 50; e == hipErrorOutOfMemory && budget_ms > 0; wait_ms *= 2) {
    const long ms = std::min(wait_ms, budget_ms);
    usleep((useconds_t)(ms * 1000));
    budget_ms -= ms;
    e = hipHostMalloc(p, bytes, flags);
  }
  return e;
}

// Workgroups for the HBM-bound kernels, measured best on MI355X (256 CUs):
// the gather (random reads, sequential writes) peaks with 2 workgroups per
// CU, the scatter (sequential reads, random writes) with one per CU: more
// random writes in flight lower its rate.  EA_GRID_HBM sets both.
// Unit order of the HBM gather / scatter: EA_HBM_ORDER=layer walks every
// entry of one layer before the next layer; the default walks each page's
// layers in turn.
int32_t hbm_layer_major(int dir) {
  const char *v = std::getenv(dir == ea::kToSlots ? "EA_GATHER_ORDER" : "EA_SCATTER_ORDER");
  if (!v || !*v) v = std::getenv("EA_HBM_ORDER");
  return v && std::strcmp(v, "layer") == 0 ? 1 : 0;
}

// Page ids of HBM copies with identity slots in the kernel arguments
// (default), or through the index ring (EA_HBM_INDEX=ring).
bool hbm_arg_pages() {
  const char *v = std::getenv("EA_HBM_INDEX");
  return !(v && std::strcmp(v, "ring") == 0);
}

int64_t grid_hbm(int dir) {
  const int both = env_int("EA_GRID_HBM", 0);
  if (dir == ea::kToSlots) return std::max(1, env_int("EA_GRID_GATHER", both ? both : 512));
  return std::max(1, env_int("EA_GRID_SCATTER", both ? both : 256));
}

// Host-link kernels: 8 workgroups (32 waves) per direction already reach the
// pinned-copy peak one way.  With a store and a load in flight together,
// more waves lower the sum (posted writes and read requests queue behind one
// another), and keeping the two directions on different XCDs raised the
// duplex sum from 63 to 87 GB/s in measurements on MI355X; spreading each
// direction's 8 workgroups over two XCDs (four on each) raised it to 89 and
// the store alone from 55.3 to 56.0 GB/s, while four XCDs (two on each)
// lowered both.  The store runs on XCDs 0 and 2 and the load on 1 and 3 by
// default (EA_XCD_STORE / EA_XCD_LOAD override the masks).  EA_LINK_WG sets
// both directions' workgroups, EA_LINK_WG_STORE / EA_LINK_WG_LOAD one each.
//
// Both directions get 8.  A ninth load workgroup carries the load to 95-96%
// of the pinned host-to-device peak during the turn's duplex whatever the
// store does, and costs the duplex 3-5%; with 8 the store's yield
// (EA_LOAD_PRIORITY below) sets the share.
int64_t grid_link(int dir) {
  const int both = env_int("EA_LINK_WG", 0);
  const int dflt = both > 0 ? both : 8;
  return std::max(1, env_int(dir == ea::kToSlots ? "EA_LINK_WG_STORE" : "EA_LINK_WG_LOAD", dflt));
}

// XCDs of the device (workgroups are dispatched round-robin over them) and
// whether kernels may place work by the XCD the hardware reports: a probe,
// run once per device when a cache first asks for hardware placement,
// checks that dispatches go round-robin over the reported XCDs (hw: -1 not
// probed yet, 0 no, 1 yes).
struct XcdInfo {
  int num = 0;
  int hw = -1;
};

XcdInfo device_xcds(int dev, bool want_hw) {
  static std::mutex mu;
  static XcdInfo known[64];
  std::lock_guard<std::mutex> lk(mu);
  if (dev < 0 || dev >= 64) return XcdInfo{1, 0};
  XcdInfo &k = known[dev];
  if (k.num == 0) {
    int v = 0, cus = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeNumberOfXccs, dev) != hipSuccess) v = 1;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      cus = 0;
    // a value that cannot be right (or a runtime without the attribute)
    // falls back to one XCD: no placement, every workgroup works
    if (v < 1 || v > 16 || cus <= 0 || cus % v != 0) v = 1;
    k.num = v;
    if (v == 1) k.hw = 0;
  }
  if (want_hw && k.hw < 0) {
    bool ok = false;
    if (ea::probe_xcd_round_robin(k.num, &ok) != hipSuccess) ok = false;
    k.hw = ok ? 1 : 0;
  }
  return k;
}

// EA_XCD_PLACEMENT=index: caches created while it is set place work by
// workgroup index instead of the XCD the hardware reports.
bool placement_by_index() {
  const char *pl = std::getenv("EA_XCD_PLACEMENT");
  return pl && std::strcmp(pl, "index") == 0;
}

uint32_t all_xcds(int n) { return n >= 32 ? 0xffffffffu : ((1u << n) - 1u); }

uint32_t xcd_mask_from_env(const char *name, uint32_t dflt, int n) {
  const char *v = std::getenv(name);
  uint32_t m = v && *v ? (uint32_t)std::strtoul(v, nullptr, 0) : dflt;
  m &= all_xcds(n);
  return m ? m : all_xcds(n);
}

bool aligned(const void *p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

// True when the n values are pairwise distinct.
template <typename T>
bool all_distinct(const T *v, int64_t n) {
  if (n <= 64) {
    for (int64_t i = 0; i < n; ++i)
      for (int64_t j = i + 1; j < n; ++j)
        if (v[i] == v[j]) return false;
    return true;
  }
  std::vector<T> s(v, v + n);
  std::sort(s.begin(), s.end());
  return std::adjacent_find(s.begin(), s.end()) == s.end();
}

// Index arrays reach the kernels through a ring of mapped, coherent pinned
// regions: the host writes region r and the kernels read it in place over
// the link (one 64-entry vector load per wave per 64 units), with no DMA
// and no device copy.  That measured 1-2% faster on MI355X than uploading
// each call's indices into a device twin first.  Region r is rewritten only
// after the event recorded behind its last consumer has fired, so
// back-to-back calls never wait on each other unless kRegions calls are
// still in flight.  The events only tell the host that the kernels have
// finished reading, so they skip the system-scope release.
class IndexRing {
 public:
  static constexpr int kRegions = 4;

  // Write slots (may be null) and pages of n entries into the next region;
  // returns their device addresses.
  int upload(const int64_t *slots, const int32_t *pages, int64_t n,
             const int64_t **d_slots, const int32_t **d_pages, int *region) {
    EA_TRY(reserve(n));
    const int r = next_;
    next_ = (next_ + 1) % kRegions;
    if (used_[r]) EA_HIP(hipEventSynchronize(ev_[r]));
    if (slots) std::memcpy(h_[r], slots, (size_t)n * 8);
    std::memcpy(h_[r] + n * 8, pages, (size_t)n * 4);
    *d_slots = reinterpret_cast<const int64_t *>(d_[r]);
    *d_pages = reinterpret_cast<const int32_t *>(d_[r] + n * 8);
    *region = r;
    return EA_OK;
  }

  // Mark the end of the region's consumers on stream s.
  int release(int r, hipStream_t s) {
    EA_HIP(hipEventRecord(ev_[r], s));
    used_[r] = true;
    return EA_OK;
  }

  void destroy() {
    for (int r = 0; r < kRegions; ++r) {
      if (ev_[r]) {
        (void)hipEventSynchronize(ev_[r]);
        (void)hipEventDestroy(ev_[r]);
      }
      if (h_[r]) (void)hipHostFree(h_[r]);
      ev_[r] = nullptr;
      h_[r] = d_[r] = nullptr;
      used_[r] = false;
    }
    cap_ = 0;
  }

 private:
  int reserve(int64_t n) {
    if (n <= cap_) return EA_OK;
    for (int r = 0; r < kRegions; ++r) {
      if (used_[r]) EA_HIP(hipEventSynchronize(ev_[r]));
      if (h_[r]) (void)hipHostFree(h_[r]);
      h_[r] = d_[r] = nullptr;
      used_[r] = false;
    }
    cap_ = 0;
    const int64_t cap = std::max<int64_t>(n, 4096);
    for (int r = 0; r < kRegions; ++r) {
      EA_HIP(hipHostMalloc((void **)&h_[r], (size_t)cap * 12,
                           hipHostMallocMapped | hipHostMallocCoherent));
      EA_HIP(hipHostGetDevicePointer((void **)&d_[r], h_[r], 0));
      if (!ev_[r]) EA_HIP(hipEventCreateWithFlags(&ev_[r], ea::kDeviceEventFlags));
    }
    cap_ = cap;
    return EA_OK;
  }

  int64_t cap_ = 0;
  uint8_t *h_[kRegions] = {};
  uint8_t *d_[kRegions] = {};
  hipEvent_t ev_[kRegions] = {};  // last consumer of the region done
  bool used_[kRegions] = {};
  int next_ = 0;
};

}  // namespace

namespace ea {
void set_last_hip(int err) { g_last_hip = err; }
}  // namespace ea

// ------------------------------------------------------------------ cache

struct ea_cache {
  ea_cache_desc d;
  int device;
  int64_t piece, page, trailer, slot;
  int32_t num_xcd;
  int32_t hw_xcd;
  std::mutex mu;  // guards the gather/scatter index ring
  IndexRing ring;
};

// ------------------------------------------------------------------- tier

namespace {

// Per-direction resources of a tier: index ring and HBM staging.  The
// staged plan double-buffers: the gather or scatter of one half runs on the
// caller's stream while the DMA copies of the other half run on the tier's
// own copy stream; events hand each half between the two.
struct DirRes {
  IndexRing ring;
  uint8_t *staging = nullptr;  // two halves of per_half slots
  int64_t per_half = 0;
  hipStream_t dma = nullptr;          // library-owned stream of the copies
  hipEvent_t start = nullptr;         // the caller's stream reached the call
  hipEvent_t ready[2] = {};           // half filled (gathered, or copied in)
  hipEvent_t done[2] = {};            // half's last user finished with it
  bool used[2] = {};
};

// The end of one transfer call: its event, the stream it was recorded on
// and the call's sequence number (0: never used).
struct EvRec {
  hipEvent_t ev = nullptr;
  hipStream_t stream = nullptr;
  int64_t seq = 0;
};

// Transfer events per tier.  Events are a bounded resource of the driver
// (each one holds a kernel event slot, a few thousand per process), so a
// tier keeps a ring of this many and never one per slot: call q uses entry
// q mod kTransferEvents, after the host has seen call q - kTransferEvents
// complete.
constexpr int64_t kTransferEvents = 64;

}  // namespace

struct ea_tier {
  std::mutex mu;
  int device = 0;
  int32_t num_layers = 0;
  int32_t has_scales = 0;
  int32_t chunk = 1;  // pages per slot
  int64_t piece = 0, page = 0, payload = 0, trailer = 0, slot = 0;
  int64_t K = 0, capacity_bytes = 0;
  uint8_t *host = nullptr;
  uint8_t *dev = nullptr;
  std::unique_ptr<ea::TierMeta> meta;
  int plan[2] = {EA_PLAN_AUTO, EA_PLAN_AUTO};
  DirRes res[2];
  std::vector<int64_t> slot_seq;  // sequence number of each slot's last transfer, 0 none
  EvRec evs[kTransferEvents];
  int64_t seq = 0;                // transfer calls so far
  int64_t bytes_stored = 0, bytes_loaded = 0, store_calls = 0, load_calls = 0;
  int64_t grid_store = 8, grid_load = 8, grid_layered = 16, grid_gather = 512, grid_scatter = 256;
  int32_t num_xcd = 1;
  uint32_t xcd_store = 1, xcd_load = 1;
  // loads have priority on the host link when yield_units > 0: load waves
  // count themselves in d_busy, and direct stores sleep while it is > 0
  uint32_t *d_busy = nullptr;
  int32_t yield_units = 0;
  int32_t controllers = 0;  // attached admission controllers (guarded by mu)
  int32_t steady_users = 0; // attached steady-clock controllers (guarded by mu)
};

namespace {

int resolve_plan(const ea_tier *t, int dir) {
  int p = t->plan[dir];
  if (p != EA_PLAN_AUTO) return p;
  const char *v = std::getenv("EA_TRANSFER");
  if (v && std::strcmp(v, "direct") == 0) return EA_PLAN_DIRECT;
  if (v && std::strcmp(v, "staged") == 0) return EA_PLAN_STAGED;
  // Measured on MI355X for every size class the workloads use (1.5 MiB
  // and 384 KiB pages, 24 MiB chunks, 768 KiB fp8 pages with scales, calls
  // of 1-8 pages of 2 MiB), both directions, consecutive and random slots:
  // the direct kernels are never slower than staging plus DMA, and are up
  // to 5x faster for single pages and 3x for random 768 KiB slots.
  return EA_PLAN_DIRECT;
}

int device_copy_stream(int dev, hipStream_t *out) {
  static std::mutex mu;
  static hipStream_t streams[64];
  if (dev < 0 || dev >= 64) return EA_EINVAL;
  std::lock_guard<std::mutex> lk(mu);
  if (!streams[dev]) EA_HIP(hipStreamCreateWithFlags(&streams[dev], hipStreamNonBlocking));
  *out = streams[dev];
  return EA_OK;
}

int ensure_staging(ea_tier *t, int dir) {
  DirRes &R = t->res[dir];
  if (R.staging) return EA_OK;
  const int64_t half = ((int64_t)env_int("EA_STAGING_MB", 512) << 20) / 2;
  const int64_t per_half = std::max<int64_t>(1, half / t->slot);
  if (!R.start) EA_HIP(hipEventCreateWithFlags(&R.start, hipEventDisableTiming));
  for (int h = 0; h < 2; ++h) {
    if (!R.ready[h]) EA_HIP(hipEventCreateWithFlags(&R.ready[h], hipEventDisableTiming));
    if (!R.done[h]) EA_HIP(hipEventCreateWithFlags(&R.done[h], hipEventDisableTiming));
  }
  // only loads copy on a stream of their own (see copy_staged): one per
  // device for the life of the process, shared by every tier (streams are
  // a runtime resource: creating one per tier and destroying it with the
  // tier churns them)
  if (dir == EA_DIR_LOAD && !R.dma) EA_TRY(device_copy_stream(t->device, &R.dma));
  EA_HIP(hipMalloc((void **)&R.staging, (size_t)(2 * per_half * t->slot)));
  R.per_half = per_half;
  return EA_OK;
}

// Order `s` after earlier transfers on other streams that touch these slots.
// A slot whose last transfer is older than the ring holds is complete: the
// host saw it finish before its event was used again.
int wait_slot_hazards(ea_tier *t, const int64_t *slots, int64_t n, hipStream_t s) {
  std::vector<int64_t> waits;
  for (int64_t i = 0; i < n; ++i) {
    const int64_t q = t->slot_seq[slots[i]];
    if (q == 0 || q <= t->seq - kTransferEvents) continue;
    const EvRec &r = t->evs[q % kTransferEvents];
    if (r.stream == s) continue;
    if (std::find(waits.begin(), waits.end(), q) == waits.end()) waits.push_back(q);
  }
  for (int64_t q : waits) {
    hipEvent_t ev = t->evs[q % kTransferEvents].ev;
    const hipError_t e = hipEventQuery(ev);
    if (e == hipSuccess) continue;
    if (e != hipErrorNotReady) {
      g_last_hip = (int)e;
      return EA_EHIP;
    }
    EA_HIP(hipStreamWaitEvent(s, ev, 0));
  }
  return EA_OK;
}

// Record the end of this call's transfer on `s` as the slots' last event.
int note_slot_transfer(ea_tier *t, const int64_t *slots, int64_t n, hipStream_t s) {
  const int64_t q = t->seq + 1;
  EvRec &r = t->evs[q % kTransferEvents];
  if (!r.ev) EA_HIP(hipEventCreateWithFlags(&r.ev, hipEventDisableTiming));
  // the entry's previous call (kTransferEvents calls ago) must be done
  // before its event is recorded again; it normally finished long ago
  if (r.seq != 0) EA_HIP(hipEventSynchronize(r.ev));
  EA_HIP(hipEventRecord(r.ev, s));
  r.stream = s;
  r.seq = q;
  t->seq = q;
  for (int64_t i = 0; i < n; ++i) t->slot_seq[slots[i]] = q;
  return EA_OK;
}

bool same_shape(const ea_tier *t, const ea_cache *c) {
  return c->d.num_layers == t->num_layers && c->piece == t->piece &&
         (c->d.scale_base != nullptr) == (t->has_scales != 0);
}

// A piece copy between the cache and buffers of slots that hold `chunk`
// pages each (chunk 1 for the cache-level gather/scatter).
ea::PieceCopy base_copy(const ea_cache *c, int64_t slot_bytes, int32_t chunk) {
  ea::PieceCopy a{};
  a.cache = static_cast<uint8_t *>(c->d.base);
  a.scales = static_cast<uint8_t *>(c->d.scale_base);
  a.num_pages = c->d.num_pages;
  a.piece_bytes = c->piece;
  a.slot_bytes = slot_bytes;
  a.payload_bytes = c->page * chunk;
  a.chunk = chunk;
  a.num_layers = c->d.num_layers;
  a.layer_begin = 0;
  a.layer_count = c->d.num_layers;
  a.num_xcd = c->num_xcd;
  a.xcd_mask = all_xcds(c->num_xcd);
  a.hw_xcd = c->hw_xcd;
  return a;
}

// Launch a piece copy for n (slot, page) entries, one per page (slots null:
// entry i goes to slot i / a.chunk): small batches carry their indices in
// the kernel arguments, and so do the page ids of HBM copies of up to
// kArgPagesMax pages with identity slots; larger ones go through the index
// ring.
int launch_entries(ea::PieceCopy a, IndexRing &ring, const int64_t *slots,
                   const int32_t *pages, int64_t n, int dir, int route, int64_t grid,
                   hipStream_t s) {
  a.n = n;
  if (n <= ea::kInlineMax) {
    ea::InlineIdx inl;
    for (int64_t i = 0; i < n; ++i) {
      inl.pages[i] = pages[i];
      inl.slots[i] = slots ? slots[i] : i / a.chunk;
    }
    EA_HIP(ea::launch_piece_copy(a, &inl, nullptr, dir, route, grid, s));
    return EA_OK;
  }
  if (route == ea::kRouteHbm && !slots && n <= ea::kArgPagesMax && hbm_arg_pages()) {
    ea::ArgPages ids;
    std::memcpy(ids.pages, pages, (size_t)n * 4);
    std::memset(ids.pages + n, 0, (size_t)(ea::kArgPagesMax - n) * 4);
    a.identity_slots = 1;
    a.pages = nullptr;
    a.slot_idx = nullptr;
    EA_HIP(ea::launch_piece_copy(a, nullptr, &ids, dir, route, grid, s));
    return EA_OK;
  }
  int region;
  EA_TRY(ring.upload(slots, pages, n, &a.slot_idx, &a.pages, &region));
  a.identity_slots = slots ? 0 : 1;
  EA_HIP(ea::launch_piece_copy(a, nullptr, nullptr, dir, route, grid, s));
  return ring.release(region, s);
}

// Direct plan: one kernel between the cache and the mapped pinned slots.
// n entries, one per page; slots[i] is the slot of page entry i.
int copy_direct(ea_tier *t, ea_cache *c, const int64_t *slots, const int32_t *pages,
                int64_t n, int dir, hipStream_t s) {
  ea::PieceCopy a = base_copy(c, t->slot, t->chunk);
  a.slots = t->dev;
  a.xcd_mask = dir == ea::kToSlots ? t->xcd_store : t->xcd_load;
  const int res_dir = dir == ea::kToSlots ? EA_DIR_STORE : EA_DIR_LOAD;
  if (t->d_busy != nullptr) {
    a.link_flag = t->d_busy;
    a.link_role = dir == ea::kToSlots ? ea::kLinkYield : ea::kLinkMark;
    a.yield_units = t->yield_units;
  }
  return launch_entries(a, t->res[res_dir].ring, slots, pages, n, dir, ea::kRouteHostLink,
                        dir == ea::kToSlots ? t->grid_store : t->grid_load, s);
}

// Staged plan: HBM staging + DMA copies of runs of consecutive slots.
// n slots (slots[i] holds pages[i*C .. i*C+C-1]); slots are processed in
// increasing order so that consecutive slots coalesce into one DMA.  The
// staging halves alternate.  A load double-buffers: the tier's copy stream
// moves one half across the link (the runtime puts these host-to-device
// copies on its copy engines) while the caller's stream scatters the other.
// A store does not: its device-to-host copies run as the runtime's blit
// kernels, and a gather running beside them holds the compute units they
// need (measured on MI355X: the 2,000-page store fell from 55.7 to 30.4
// GB/s with its copies on a second stream), so gather and copies take
// turns on the caller's stream.
int copy_staged(ea_tier *t, ea_cache *c, const int64_t *slots, const int32_t *pages,
                int64_t n, int dir, hipStream_t s) {
  const int res_dir = dir == ea::kToSlots ? EA_DIR_STORE : EA_DIR_LOAD;
  EA_TRY(ensure_staging(t, res_dir));
  DirRes &R = t->res[res_dir];
  hipStream_t cs = dir == ea::kToSlots ? s : R.dma;  // the stream of the copies
  // the copies start after everything the caller ordered before the call
  if (cs != s) {
    EA_HIP(hipEventRecord(R.start, s));
    EA_HIP(hipStreamWaitEvent(cs, R.start, 0));
  }

  const int64_t C = t->chunk;
  std::vector<int64_t> order((size_t)n);
  for (int64_t i = 0; i < n; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(),
                   [&](int64_t x, int64_t y) { return slots[x] < slots[y]; });
  std::vector<int64_t> ss((size_t)n);
  std::vector<int32_t> pp((size_t)(n * C));
  for (int64_t i = 0; i < n; ++i) {
    ss[i] = slots[order[i]];
    std::memcpy(&pp[i * C], pages + order[i] * C, (size_t)C * sizeof(int32_t));
  }
  const int64_t per = R.per_half;
  for (int64_t c0 = 0, half = 0; c0 < n; c0 += per, ++half) {
    const int64_t c1 = std::min(n, c0 + per);
    const int b = (int)(half & 1);
    uint8_t *stage = R.staging + b * per * t->slot;
    ea::PieceCopy a = base_copy(c, t->slot, t->chunk);
    a.slots = stage;
    if (dir == ea::kToSlots) {
      // gather on the caller's stream once the half's earlier copies are done
      if (R.used[b]) EA_HIP(hipStreamWaitEvent(s, R.done[b], 0));
      EA_TRY(launch_entries(a, R.ring, nullptr, pp.data() + c0 * C, (c1 - c0) * C, dir,
                            ea::kRouteHbm, t->grid_gather, s));
      if (cs != s) {
        EA_HIP(hipEventRecord(R.ready[b], s));
        EA_HIP(hipStreamWaitEvent(cs, R.ready[b], 0));
      }
    } else if (R.used[b]) {
      // copies into the half once its earlier scatter is done
      EA_HIP(hipStreamWaitEvent(cs, R.done[b], 0));
    }
    for (int64_t j0 = c0; j0 < c1;) {
      int64_t j1 = j0 + 1;
      while (j1 < c1 && ss[j1] == ss[j1 - 1] + 1) ++j1;
      uint8_t *h = t->host + ss[j0] * t->slot;
      uint8_t *g = stage + (j0 - c0) * t->slot;
      const size_t bytes = (size_t)((j1 - j0) * t->slot);
      if (dir == ea::kToSlots)
        EA_HIP(hipMemcpyAsync(h, g, bytes, hipMemcpyDeviceToHost, cs));
      else
        EA_HIP(hipMemcpyAsync(g, h, bytes, hipMemcpyHostToDevice, cs));
      j0 = j1;
    }
    if (dir == ea::kToSlots) {
      EA_HIP(hipEventRecord(R.done[b], cs));
    } else {
      EA_HIP(hipEventRecord(R.ready[b], cs));
      EA_HIP(hipStreamWaitEvent(s, R.ready[b], 0));
      EA_TRY(launch_entries(a, R.ring, nullptr, pp.data() + c0 * C, (c1 - c0) * C, dir,
                            ea::kRouteHbm, t->grid_scatter, s));
      EA_HIP(hipEventRecord(R.done[b], s));
    }
    R.used[b] = true;
  }
  return EA_OK;  // every copy and scatter ends on the caller's stream
}

int validate_cache_desc(const ea_cache_desc *d) {
  if (!d || !d->base) return EA_EINVAL;
  if (d->num_pages < 1 || d->num_layers < 1 || d->page_tokens < 1 || d->num_kv_heads < 1 ||
      d->head_dim < 1 || d->elem_bytes < 1)
    return EA_EINVAL;
  const int64_t piece = 2LL * d->page_tokens * d->num_kv_heads * d->head_dim * d->elem_bytes;
  if (piece % 16 != 0) return EA_EINVAL;
  if (!aligned(d->base, 16)) return EA_EINVAL;
  if (d->scale_base && !aligned(d->scale_base, 8)) return EA_EINVAL;
  return EA_OK;
}

// n slots, n * C destination pages (all distinct).
int validate_load(ea_tier *t, ea_cache *c, const int64_t *host_slots,
                  const int32_t *dst_pages, int32_t n) {
  if (!c || !t || n < 0) return EA_EINVAL;
  if (!same_shape(t, c)) return EA_EINVAL;
  if (n == 0) return EA_OK;
  if (!host_slots || !dst_pages) return EA_EINVAL;
  if ((int64_t)n * t->chunk > INT32_MAX) return EA_EINVAL;
  const int64_t m = (int64_t)n * t->chunk;
  for (int32_t i = 0; i < n; ++i)
    if (host_slots[i] < 0 || host_slots[i] >= t->K) return EA_EINVAL;
  for (int64_t i = 0; i < m; ++i)
    if (dst_pages[i] < 0 || dst_pages[i] >= c->d.num_pages) return EA_EINVAL;
  if (!all_distinct(dst_pages, m)) return EA_EINVAL;
  return EA_OK;
}

// The slot of every page entry: slot i repeated C times.
std::vector<int64_t> per_page_slots(const int64_t *slots, int64_t n, int64_t C) {
  std::vector<int64_t> v((size_t)(n * C));
  for (int64_t i = 0; i < n; ++i)
    for (int64_t c = 0; c < C; ++c) v[(size_t)(i * C + c)] = slots[i];
  return v;
}

}  // namespace

extern "C" {

const char *ea_strerror(int code) {
  switch (code) {
    case EA_OK: return "ok";
    case EA_EINVAL: return "invalid argument";
    case EA_ENOMEM: return "out of memory";
    case EA_ENOSPC: return "no space";
    case EA_EHIP: return "HIP runtime error";
    case EA_ENOTSUP: return "not supported";
    default: return "unknown error";
  }
}

int ea_last_hip_error(void) { return g_last_hip; }

int ea_cache_create(const ea_cache_desc *desc, ea_cache **out) {
  if (!out) return EA_EINVAL;
  EA_TRY(validate_cache_desc(desc));
  int dev;
  EA_HIP(hipGetDevice(&dev));
  ea_cache *c = new (std::nothrow) ea_cache;
  if (!c) return EA_ENOMEM;
  c->d = *desc;
  c->device = dev;
  const bool want_hw = !placement_by_index();
  const XcdInfo xi = device_xcds(dev, want_hw);
  c->num_xcd = xi.num;
  c->hw_xcd = want_hw && xi.hw == 1 ? 1 : 0;
  c->piece = 2LL * desc->page_tokens * desc->num_kv_heads * desc->head_dim * desc->elem_bytes;
  c->page = c->piece * desc->num_layers;
  c->trailer = desc->scale_base ? ((int64_t)desc->num_layers * 8 + 255) / 256 * 256 : 0;
  c->slot = c->page + c->trailer;
  *out = c;
  return EA_OK;
}

int ea_cache_destroy(ea_cache *cache) {
  if (!cache) return EA_EINVAL;
  {
    DeviceScope ds(cache->device);
    std::lock_guard<std::mutex> lk(cache->mu);
    cache->ring.destroy();
  }
  delete cache;
  return EA_OK;
}

int ea_tier_create(const ea_cache *shape, int64_t capacity_bytes, int numa_node,
                   ea_tier **out) {
  return ea_tier_create_chunked(shape, 1, capacity_bytes, numa_node, out);
}

int ea_tier_create_chunked(const ea_cache *shape, int32_t chunk_pages, int64_t capacity_bytes,
                           int numa_node, ea_tier **out) {
  try {
    if (!shape || !out || capacity_bytes <= 0 || chunk_pages < 1) return EA_EINVAL;
    const int64_t payload = shape->page * chunk_pages;
    const int64_t trailer =
        shape->d.scale_base ? ((int64_t)shape->d.num_layers * chunk_pages * 8 + 255) / 256 * 256 : 0;
    const int64_t slot_bytes = payload + trailer;
    const int64_t K = capacity_bytes / slot_bytes;
    if (K < 1) return EA_EINVAL;
    DeviceScope ds(shape->device);
    EA_TRY(ds.status());
    std::unique_ptr<ea_tier> t(new (std::nothrow) ea_tier);
    if (!t) return EA_ENOMEM;
    t->device = shape->device;
    t->num_layers = shape->d.num_layers;
    t->has_scales = shape->d.scale_base != nullptr;
    t->chunk = chunk_pages;
    t->piece = shape->piece;
    t->page = shape->page;
    t->payload = payload;
    t->trailer = trailer;
    t->slot = slot_bytes;
    t->K = K;
    t->capacity_bytes = capacity_bytes;
    t->grid_store = grid_link(ea::kToSlots);
    t->grid_load = grid_link(ea::kToPages);
    t->num_xcd = shape->num_xcd;
    // the two directions on different XCDs: two each (store 0 and 2, load 1
    // and 3) when the device has at least four, one each when it has two
    const int nx = t->num_xcd;
    t->xcd_store = xcd_mask_from_env("EA_XCD_STORE", nx >= 4 ? 0x5u : 0x1u, nx);
    t->xcd_load = xcd_mask_from_env("EA_XCD_LOAD", nx >= 4 ? 0xAu : (nx > 1 ? 0x2u : 0x1u), nx);
    t->grid_gather = grid_hbm(ea::kToSlots);
    t->grid_scatter = grid_hbm(ea::kToPages);
    // a layered load is one short kernel per layer: 16 workgroups hide the
    // start and drain of each (56 GB/s against 51 with 8 on MI355X)
    t->grid_layered = std::max(1, env_int("EA_LINK_WG_LAYERED", 16));
    // Fine-grained (coherent) by default: kernels and DMA engines then see one
    // another's writes to the slots without any cache maintenance.
    unsigned flags = hipHostMallocMapped | hipHostMallocPortable;
    flags |= env_int("EA_HOST_COHERENT", 1) ? hipHostMallocCoherent : hipHostMallocNonCoherent;
    bool numa_set = false;
    if (numa_node >= 0 && numa_node < 64) {
      // prefer the requested node for the pinned pages (MPOL_PREFERRED = 1)
      unsigned long mask = 1ul << numa_node;
      numa_set = syscall(SYS_set_mempolicy, 1, &mask, 64) == 0;
      if (numa_set) flags |= hipHostMallocNumaUser;
    }
    hipError_t e = host_alloc_retry((void **)&t->host, (size_t)(K * t->slot), flags);
    if (numa_set) (void)syscall(SYS_set_mempolicy, 0, nullptr, 0);
    if (e != hipSuccess) {
      g_last_hip = (int)e;
      return EA_ENOMEM;
    }
    e = hipHostGetDevicePointer((void **)&t->dev, t->host, 0);
    if (e != hipSuccess) {
      (void)hipHostFree(t->host);
      g_last_hip = (int)e;
      return EA_EHIP;
    }
    // Loads first on the host link: a restore is the T_load of Eq. 2 that a
    // waiting request pays, a store is background write-back.  While waves
    // of a load of this tier run, each wave of a direct store sleeps
    // EA_LOAD_PRIORITY x 1,024 cycles per 32 KiB it copies.  Measured on the
    // Qwen3 turn (2,000-page store beside a 1,500-page load, 8 workgroups
    // each way), load in the step / duplex: off 76% / 88.3 GB/s, 28 units
    // 77% / 88.9, 30 82% / 87.0, 32 85% / 85.2, 34 87% / 83.5, 40 90% /
    // 79.2.  31 keeps the restore above 80% of the host-to-device peak and
    // the duplex above 85 GB/s.  EA_LOAD_PRIORITY=0 turns it off.
    t->yield_units = std::max(0, env_int("EA_LOAD_PRIORITY", 31));
    if (t->yield_units > 0) {
      e = hipMalloc((void **)&t->d_busy, 256);
      if (e == hipSuccess) e = hipMemset(t->d_busy, 0, 256);
      if (e != hipSuccess) {
        if (t->d_busy) (void)hipFree(t->d_busy);
        (void)hipHostFree(t->host);
        g_last_hip = (int)e;
        return EA_EHIP;
      }
    }
    t->meta.reset(new (std::nothrow) ea::TierMeta(K, capacity_bytes));
    if (!t->meta) {
      if (t->d_busy) (void)hipFree(t->d_busy);
      (void)hipHostFree(t->host);
      return EA_ENOMEM;
    }
    t->slot_seq.assign((size_t)K, 0);
    *out = t.release();
    return EA_OK;
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
}

int ea_tier_destroy(ea_tier *t) {
  if (!t) return EA_EINVAL;
  {
    std::lock_guard<std::mutex> lk(t->mu);
    if (t->controllers > 0) return EA_EINVAL;  // a controller still uses it
  }
  {
    DeviceScope ds(t->device);
    std::lock_guard<std::mutex> lk(t->mu);
    for (auto &ev : t->evs)
      if (ev.ev) {
        (void)hipEventSynchronize(ev.ev);
        (void)hipEventDestroy(ev.ev);
      }
    for (auto &R : t->res) {
      R.ring.destroy();
      // the device's copy stream outlives the tier; its events below
      // cover this tier's copies on it
      for (hipEvent_t e : {R.start, R.ready[0], R.ready[1], R.done[0], R.done[1]})
        if (e) {
          (void)hipEventSynchronize(e);
          (void)hipEventDestroy(e);
        }
      if (R.staging) (void)hipFree(R.staging);
    }
    if (t->host) (void)hipHostFree(t->host);
    if (t->d_busy) (void)hipFree(t->d_busy);
  }
  delete t;
  return EA_OK;
}

}  // extern "C"

void ea::tier_use_steady_clock(ea_tier *t, bool on) {
  std::lock_guard<std::mutex> lk(t->mu);
  // one count per steady-clock controller: the tier keeps the steady clock
  // until the last of them detaches
  t->steady_users += on ? 1 : -1;
  t->meta->use_steady_clock(t->steady_users > 0);
}

void ea::tier_attach_controller(ea_tier *t, int delta) {
  std::lock_guard<std::mutex> lk(t->mu);
  t->controllers += delta;
}

extern "C" {

int ea_tier_get_info(const ea_tier *t, ea_tier_info *info) {
  if (!t || !info) return EA_EINVAL;
  info->capacity_slots = t->K;
  info->slot_bytes = t->slot;
  info->piece_bytes = t->piece;
  info->page_bytes = t->payload;
  info->trailer_bytes = t->trailer;
  info->capacity_bytes = t->capacity_bytes;
  info->host_base = t->host;
  info->device_base = t->dev;
  info->chunk_pages = t->chunk;
  return EA_OK;
}

int ea_tier_lookup(ea_tier *t, const uint8_t *keys, int64_t n, int64_t *hit_blocks,
                   int64_t *slots_out) {
  try {
    if (!t || n < 0 || !hit_blocks) return EA_EINVAL;
    if (n > 0 && (!keys || !slots_out)) return EA_EINVAL;
    std::lock_guard<std::mutex> lk(t->mu);
    return t->meta->lookup(keys, n, hit_blocks, slots_out);
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
}

int ea_admission_fill(ea_tier *t, const ea_policy *p, const ea_request *r,
                      const uint8_t *keys, int64_t n_keys, uint8_t *mask_out,
                      int32_t *save_out) {
  try {
    if (!t || !p || !r || !save_out || n_keys < 0) return EA_EINVAL;
    if (n_keys > 0 && (!keys || !mask_out)) return EA_EINVAL;
    std::lock_guard<std::mutex> lk(t->mu);
    return t->meta->admission(*p, *r, keys, n_keys, mask_out, save_out);
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
}

int ea_admission_fill_report(ea_tier *t, const ea_policy *p, const ea_request *r,
                             const ea_tier_report *report, int64_t max_age,
                             const uint8_t *keys, int64_t n_keys, uint8_t *mask_out,
                             int32_t *save_out) {
  try {
    if (!t || !p || !r || !save_out || n_keys < 0 || max_age < 0) return EA_EINVAL;
    if (n_keys > 0 && (!keys || !mask_out)) return EA_EINVAL;
    std::lock_guard<std::mutex> lk(t->mu);
    return t->meta->admission(*p, *r, keys, n_keys, mask_out, save_out, true, report, max_age);
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
}

int ea_tier_publish(ea_tier *t, int64_t now, int64_t window, ea_tier_report *out) {
  try {
    if (!t || !out) return EA_EINVAL;
    std::lock_guard<std::mutex> lk(t->mu);
    return t->meta->publish(now, window, out);
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
}

int ea_tier_alloc(ea_tier *t, const uint8_t *keys, const uint8_t *mask, int64_t n,
                  int64_t *slots_out, int64_t *allocated) {
  try {
    if (!t || n < 0 || !allocated) return EA_EINVAL;
    if (n > 0 && (!keys || !slots_out)) return EA_EINVAL;
    std::lock_guard<std::mutex> lk(t->mu);
    return t->meta->alloc(keys, mask, n, slots_out, allocated);
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
}

int ea_tier_unpin(ea_tier *t, const int64_t *slots, int64_t n) {
  try {
    if (!t || n < 0) return EA_EINVAL;
    if (n == 0) return EA_OK;
    if (!slots) return EA_EINVAL;
    std::lock_guard<std::mutex> lk(t->mu);
    return t->meta->unpin(slots, n);
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
}

int ea_tier_stats(const ea_tier *t, ea_tier_stats_t *s) {
  if (!t || !s) return EA_EINVAL;
  std::memset(s, 0, sizeof *s);
  std::lock_guard<std::mutex> lk(const_cast<ea_tier *>(t)->mu);
  t->meta->stats(s);
  s->bytes_stored = t->bytes_stored;
  s->bytes_loaded = t->bytes_loaded;
  s->store_calls = t->store_calls;
  s->load_calls = t->load_calls;
  return EA_OK;
}

int ea_tier_export(const ea_tier *t, uint8_t *state_out, int32_t *pins_out,
                   uint8_t *keys_out, int64_t *lru_out, int64_t *n_lru) {
  if (!t || !state_out || !pins_out || !keys_out || !lru_out || !n_lru) return EA_EINVAL;
  std::lock_guard<std::mutex> lk(const_cast<ea_tier *>(t)->mu);
  t->meta->export_state(state_out, pins_out, keys_out, lru_out, n_lru);
  return EA_OK;
}

int ea_tier_set_plan(ea_tier *t, int direction, int plan) {
  if (!t || plan < EA_PLAN_AUTO || plan > EA_PLAN_STAGED) return EA_EINVAL;
  if (direction < EA_DIR_STORE || direction > EA_DIR_BOTH) return EA_EINVAL;
  std::lock_guard<std::mutex> lk(t->mu);
  if (direction != EA_DIR_LOAD) t->plan[EA_DIR_STORE] = plan;
  if (direction != EA_DIR_STORE) t->plan[EA_DIR_LOAD] = plan;
  return EA_OK;
}

int ea_tier_get_plan(const ea_tier *t, int direction, int *plan) {
  if (!t || !plan || (direction != EA_DIR_STORE && direction != EA_DIR_LOAD)) return EA_EINVAL;
  *plan = resolve_plan(t, direction);
  return EA_OK;
}

int ea_store_blocks(ea_cache *c, ea_tier *t, const int32_t *block_ids,
                    const int64_t *host_slots, const uint8_t *admit_mask, int32_t n,
                    hipStream_t stream) {
  try {
    if (!c || !t || n < 0) return EA_EINVAL;
    if (!same_shape(t, c)) return EA_EINVAL;
    if (n == 0) return EA_OK;
    if (!block_ids || !host_slots) return EA_EINVAL;
    const int64_t C = t->chunk;
    if ((int64_t)n * C > INT32_MAX) return EA_EINVAL;
    std::vector<int64_t> slots;
    std::vector<int32_t> pages;
    slots.reserve((size_t)n);
    pages.reserve((size_t)(n * C));
    for (int32_t i = 0; i < n; ++i) {
      if (admit_mask && !admit_mask[i]) continue;
      if (host_slots[i] < 0 || host_slots[i] >= t->K) return EA_EINVAL;
      for (int64_t k = 0; k < C; ++k) {
        const int32_t p = block_ids[i * C + k];
        if (p < 0 || p >= c->d.num_pages) return EA_EINVAL;
        pages.push_back(p);
      }
      slots.push_back(host_slots[i]);
    }
    const int64_t m = (int64_t)slots.size();
    if (!all_distinct(slots.data(), m)) return EA_EINVAL;
    if (m == 0) return EA_OK;
    DeviceScope ds(t->device);
    EA_TRY(ds.status());
    std::lock_guard<std::mutex> lk(t->mu);
    EA_TRY(wait_slot_hazards(t, slots.data(), m, stream));
    if (resolve_plan(t, EA_DIR_STORE) == EA_PLAN_STAGED) {
      EA_TRY(copy_staged(t, c, slots.data(), pages.data(), m, ea::kToSlots, stream));
    } else {
      const std::vector<int64_t> each = per_page_slots(slots.data(), m, C);
      EA_TRY(copy_direct(t, c, each.data(), pages.data(), m * C, ea::kToSlots, stream));
    }
    EA_TRY(note_slot_transfer(t, slots.data(), m, stream));
    for (int64_t i = 0; i < m; ++i) t->meta->mark_stored(slots[i]);
    t->bytes_stored += m * t->slot;
    t->store_calls += 1;
    return EA_OK;
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
}

int ea_load_blocks(ea_tier *t, ea_cache *c, const int64_t *host_slots,
                   const int32_t *dst_pages, int32_t n, hipStream_t stream) {
  try {
    EA_TRY(validate_load(t, c, host_slots, dst_pages, n));
    if (n == 0) return EA_OK;
    DeviceScope ds(t->device);
    EA_TRY(ds.status());
    std::lock_guard<std::mutex> lk(t->mu);
    EA_TRY(wait_slot_hazards(t, host_slots, n, stream));
    if (resolve_plan(t, EA_DIR_LOAD) == EA_PLAN_STAGED) {
      EA_TRY(copy_staged(t, c, host_slots, dst_pages, n, ea::kToPages, stream));
    } else {
      const std::vector<int64_t> each = per_page_slots(host_slots, n, t->chunk);
      EA_TRY(copy_direct(t, c, each.data(), dst_pages, (int64_t)n * t->chunk, ea::kToPages,
                         stream));
    }
    EA_TRY(note_slot_transfer(t, host_slots, n, stream));
    t->bytes_loaded += (int64_t)n * t->slot;
    t->load_calls += 1;
    return EA_OK;
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
}

int ea_load_blocks_layered(ea_tier *t, ea_cache *c, const int64_t *host_slots,
                           const int32_t *dst_pages, int32_t n, hipStream_t copy_stream,
                           hipEvent_t *layer_done, int32_t n_events) {
  try {
    if (!layer_done || !c || n_events != c->d.num_layers) return EA_EINVAL;
    EA_TRY(validate_load(t, c, host_slots, dst_pages, n));
    for (int32_t l = 0; l < c->d.num_layers; ++l)
      if (!layer_done[l]) return EA_EINVAL;
    DeviceScope ds(t->device);
    EA_TRY(ds.status());
    std::lock_guard<std::mutex> lk(t->mu);
    if (n == 0) {
      for (int32_t l = 0; l < c->d.num_layers; ++l)
        EA_HIP(hipEventRecord(layer_done[l], copy_stream));
      return EA_OK;
    }
    EA_TRY(wait_slot_hazards(t, host_slots, n, copy_stream));
    // the pieces of one layer are strided inside the slots, so every layer is
    // its own direct kernel over all n slots
    const int64_t m = (int64_t)n * t->chunk;  // page entries
    const std::vector<int64_t> each = per_page_slots(host_slots, n, t->chunk);
    ea::PieceCopy a = base_copy(c, t->slot, t->chunk);
    a.slots = t->dev;
    a.xcd_mask = t->xcd_load;
    a.n = m;
    a.layer_count = 1;
    ea::InlineIdx inl;
    const ea::InlineIdx *pin = nullptr;
    IndexRing &ring = t->res[EA_DIR_LOAD].ring;
    int region = -1;
    if (m <= ea::kInlineMax) {
      for (int64_t i = 0; i < m; ++i) {
        inl.pages[i] = dst_pages[i];
        inl.slots[i] = each[(size_t)i];
      }
      pin = &inl;
    } else {
      EA_TRY(ring.upload(each.data(), dst_pages, m, &a.slot_idx, &a.pages, &region));
    }
    if (t->d_busy != nullptr) {
      a.link_flag = t->d_busy;
      a.link_role = ea::kLinkMark;
    }
    hipError_t e = hipSuccess;
    for (int32_t l = 0; l < c->d.num_layers && e == hipSuccess; ++l) {
      a.layer_begin = l;
      e = ea::launch_piece_copy(a, pin, nullptr, ea::kToPages, ea::kRouteHostLink,
                                t->grid_layered, copy_stream);
      if (e == hipSuccess) e = hipEventRecord(layer_done[l], copy_stream);
    }
    EA_HIP(e);
    if (region >= 0) EA_TRY(ring.release(region, copy_stream));
    EA_TRY(note_slot_transfer(t, host_slots, n, copy_stream));
    t->bytes_loaded += (int64_t)n * t->slot;
    t->load_calls += 1;
    return EA_OK;
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
}

// ------------------------------------------------- gather / scatter (HBM)

int ea_gather_blocks(ea_cache *c, const int32_t *block_ids, int32_t n, void *d_dst,
                     int64_t dst_bytes, hipStream_t stream) {
  try {
    if (!c || n < 0 || dst_bytes < 0) return EA_EINVAL;
    if (n == 0) return EA_OK;
    if (!block_ids || !d_dst || !aligned(d_dst, 16)) return EA_EINVAL;
    if (dst_bytes / c->slot < n) return EA_EINVAL;  // n slots must fit
    for (int32_t i = 0; i < n; ++i)
      if (block_ids[i] < 0 || block_ids[i] >= c->d.num_pages) return EA_EINVAL;
    DeviceScope ds(c->device);
    EA_TRY(ds.status());
    std::lock_guard<std::mutex> lk(c->mu);
    ea::PieceCopy a = base_copy(c, c->slot, 1);
    a.slots = static_cast<uint8_t *>(d_dst);
    a.layer_major = hbm_layer_major(ea::kToSlots);
    return launch_entries(a, c->ring, nullptr, block_ids, n, ea::kToSlots, ea::kRouteHbm,
                          grid_hbm(ea::kToSlots), stream);
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
}

int ea_scatter_blocks(ea_cache *c, const void *d_src, int64_t src_bytes,
                      const int32_t *dst_pages, int32_t n, hipStream_t stream) {
  try {
    if (!c || n < 0 || src_bytes < 0) return EA_EINVAL;
    if (n == 0) return EA_OK;
    if (!dst_pages || !d_src || !aligned(d_src, 16)) return EA_EINVAL;
    if (src_bytes / c->slot < n) return EA_EINVAL;  // n slots must be there
    for (int32_t i = 0; i < n; ++i)
      if (dst_pages[i] < 0 || dst_pages[i] >= c->d.num_pages) return EA_EINVAL;
    if (!all_distinct(dst_pages, n)) return EA_EINVAL;
    DeviceScope ds(c->device);
    EA_TRY(ds.status());
    std::lock_guard<std::mutex> lk(c->mu);
    ea::PieceCopy a = base_copy(c, c->slot, 1);
    a.slots = static_cast<uint8_t *>(const_cast<void *>(d_src));
    a.layer_major = hbm_layer_major(ea::kToPages);
    return launch_entries(a, c->ring, nullptr, dst_pages, n, ea::kToPages, ea::kRouteHbm,
                          grid_hbm(ea::kToPages), stream);
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
}

// ------------------------------------------- consumer stand-in (checksum)

int ea_layer_checksum(ea_cache *c, int32_t layer, const int32_t *pages, int32_t n,
                      uint64_t *d_out, int64_t out_capacity, hipStream_t stream) {
  try {
    if (!c || n < 0 || layer < 0 || layer >= c->d.num_layers) return EA_EINVAL;
    if (n == 0) return EA_OK;
    if (!pages || !d_out || !aligned(d_out, 8) || out_capacity < n) return EA_EINVAL;
    for (int32_t i = 0; i < n; ++i)
      if (pages[i] < 0 || pages[i] >= c->d.num_pages) return EA_EINVAL;
    DeviceScope ds(c->device);
    EA_TRY(ds.status());
    std::lock_guard<std::mutex> lk(c->mu);
    const int64_t *unused = nullptr;
    const int32_t *d_pages = nullptr;
    int region;
    EA_TRY(c->ring.upload(nullptr, pages, n, &unused, &d_pages, &region));
    EA_HIP(ea::launch_layer_checksum(static_cast<const uint8_t *>(c->d.base),
                                     static_cast<const uint8_t *>(c->d.scale_base),
                                     c->d.num_pages, c->piece, layer, d_pages, n, d_out, stream));
    return c->ring.release(region, stream);
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
}

// --------------------------------------------------------------- peak probe

int ea_peak_probe(ea_tier *t, void *d_buf, int64_t bytes, int direction, int reps,
                  double *gbps) {
  if (!t || !d_buf || !gbps || bytes <= 0 || reps < 1) return EA_EINVAL;
  if (direction < EA_DIR_STORE || direction > EA_DIR_BOTH) return EA_EINVAL;
  const int64_t need = direction == EA_DIR_BOTH ? 2 * bytes : bytes;
  if (need > t->K * t->slot) return EA_EINVAL;
  DeviceScope ds(t->device);
  EA_TRY(ds.status());
  std::lock_guard<std::mutex> lk(t->mu);
  // the probe overwrites the first slots: refuse while any of them is in use
  if (!t->meta->slots_free(0, (need + t->slot - 1) / t->slot)) return EA_EINVAL;
  for (auto &ev : t->evs)
    if (ev.ev) EA_HIP(hipEventSynchronize(ev.ev));
  hipStream_t s[2] = {nullptr, nullptr};
  hipEvent_t e0[2] = {nullptr, nullptr}, e1[2] = {nullptr, nullptr};
  int rc = EA_OK;
  double best = 0.0;
  auto fail = [&](hipError_t e) {
    g_last_hip = (int)e;
    rc = EA_EHIP;
  };
  for (int i = 0; i < 2 && rc == EA_OK; ++i) {
    hipError_t e;
    if ((e = hipStreamCreateWithFlags(&s[i], hipStreamNonBlocking)) != hipSuccess) fail(e);
    else if ((e = hipEventCreate(&e0[i])) != hipSuccess) fail(e);
    else if ((e = hipEventCreate(&e1[i])) != hipSuccess) fail(e);
  }
  uint8_t *dbuf = static_cast<uint8_t *>(d_buf);
  const int streams = direction == EA_DIR_BOTH ? 2 : 1;
  for (int r = 0; r < reps && rc == EA_OK; ++r) {
    hipError_t e = hipSuccess;
    for (int i = 0; i < streams && e == hipSuccess; ++i) {
      const bool d2h = direction == EA_DIR_STORE || (direction == EA_DIR_BOTH && i == 0);
      uint8_t *h = t->host + i * bytes;
      uint8_t *g = dbuf + i * bytes;
      e = hipEventRecord(e0[i], s[i]);
      if (e == hipSuccess)
        e = d2h ? hipMemcpyAsync(h, g, (size_t)bytes, hipMemcpyDeviceToHost, s[i])
                : hipMemcpyAsync(g, h, (size_t)bytes, hipMemcpyHostToDevice, s[i]);
      if (e == hipSuccess) e = hipEventRecord(e1[i], s[i]);
    }
    float worst = 0.f;
    for (int i = 0; i < streams && e == hipSuccess; ++i) {
      e = hipEventSynchronize(e1[i]);
      float ms = 0.f;
      if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0[i], e1[i]);
      worst = std::max(worst, ms);
    }
    if (e != hipSuccess) {
      fail(e);
      break;
    }
    best = std::max(best, (double)(streams * bytes) / (worst * 1e-3) / 1e9);
  }
  for (int i = 0; i < 2; ++i) {
    if (s[i]) (void)hipStreamSynchronize(s[i]);
    if (e0[i]) (void)hipEventDestroy(e0[i]);
    if (e1[i]) (void)hipEventDestroy(e1[i]);
    if (s[i]) (void)hipStreamDestroy(s[i]);
  }
  if (rc == EA_OK) *gbps = best;
  return rc;
}

}  // extern "C"
