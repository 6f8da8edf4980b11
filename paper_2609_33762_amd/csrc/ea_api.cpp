// C ABI of libea (include/ea.h): validation, pinned host tier, transfer
// plans, stream/event bookkeeping and the hash entry points.
#include <hip/hip_runtime_api.h>
#include <sys/syscall.h>
#include <unistd.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <memory>
#include <mutex>
#include <new>
#include <unordered_set>
#include <vector>

#include "ea.h"
#include "ea_internal.hpp"
#include "ea_tier_meta.hpp"

namespace {

thread_local int g_last_hip = 0;

#define EA_HIP(expr)                       \
  do {                                     \
    hipError_t e_ = (expr);                \
    if (e_ != hipSuccess) {                \
      g_last_hip = (int)e_;                \
      return EA_EHIP;                      \
    }                                      \
  } while (0)

#define EA_TRY(expr)          \
  do {                        \
    int rc_ = (expr);         \
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

}  // namespace

namespace ea {
void set_last_hip(int err) { g_last_hip = err; }
}  // namespace ea

// ------------------------------------------------------------------ cache

struct ea_cache {
  ea_cache_desc d;
  int device;
  int64_t piece, page, trailer, slot;
};

// ------------------------------------------------------------------- tier

namespace {

constexpr int kRegions = 2;  // index upload regions per direction

struct DirRes {
  int64_t cap = 0;  // entries per region
  uint8_t *h[kRegions] = {};
  uint8_t *d[kRegions] = {};
  hipEvent_t ev[kRegions] = {};
  bool used[kRegions] = {};
  int next = 0;
  uint8_t *staging = nullptr;  // HBM, two halves
  int64_t per_half = 0;        // slots per half
  hipEvent_t staging_ev = nullptr;
  hipStream_t staging_stream = nullptr;
  bool staging_used = false;
};

struct EvRec {
  hipEvent_t ev;
  hipStream_t stream;
  int32_t refs;
};

}  // namespace

struct ea_tier {
  std::mutex mu;
  int device = 0;
  int32_t num_layers = 0;
  int32_t has_scales = 0;
  int64_t piece = 0, page = 0, trailer = 0, slot = 0;
  int64_t K = 0, capacity_bytes = 0;
  uint8_t *host = nullptr;
  uint8_t *dev = nullptr;
  std::unique_ptr<ea::TierMeta> meta;
  int plan[2] = {EA_PLAN_AUTO, EA_PLAN_AUTO};
  DirRes res[2];
  std::vector<int32_t> slot_ev;  // last transfer event of each slot, -1 none
  std::vector<EvRec> evs;
  std::vector<int32_t> free_evs;
  int64_t bytes_stored = 0, bytes_loaded = 0, store_calls = 0, load_calls = 0;
  int grid_cap = 0;
};

namespace {

int resolve_plan(const ea_tier *t, int dir) {
  int p = t->plan[dir];
  if (p != EA_PLAN_AUTO) return p;
  const char *v = std::getenv("EA_TRANSFER");
  if (v && std::strcmp(v, "direct") == 0) return EA_PLAN_DIRECT;
  if (v && std::strcmp(v, "staged") == 0) return EA_PLAN_STAGED;
  return EA_PLAN_DIRECT;
}

int64_t default_staging_bytes() {
  return (int64_t)env_int("EA_STAGING_MB", 512) << 20;
}

// Make sure region r of direction `dir` can hold n entries (12 bytes each).
int ensure_regions(ea_tier *t, int dir, int64_t n) {
  DirRes &R = t->res[dir];
  if (n <= R.cap) return EA_OK;
  for (int r = 0; r < kRegions; ++r) {
    if (R.used[r]) EA_HIP(hipEventSynchronize(R.ev[r]));
    if (R.h[r]) (void)hipHostFree(R.h[r]);
    if (R.d[r]) (void)hipFree(R.d[r]);
    R.h[r] = R.d[r] = nullptr;
    R.used[r] = false;
  }
  int64_t cap = std::max<int64_t>(n, 4096);
  for (int r = 0; r < kRegions; ++r) {
    EA_HIP(hipHostMalloc((void **)&R.h[r], (size_t)cap * 12, hipHostMallocDefault));
    EA_HIP(hipMalloc((void **)&R.d[r], (size_t)cap * 12));
    if (!R.ev[r]) EA_HIP(hipEventCreateWithFlags(&R.ev[r], hipEventDisableTiming));
  }
  R.cap = cap;
  return EA_OK;
}

// Copy (slots, pages) to the device; returns the device arrays.
int upload_indices(ea_tier *t, int dir, const int64_t *slots,
                   const int32_t *pages, int64_t n, hipStream_t s,
                   const int64_t **d_slots, const int32_t **d_pages, int *region) {
  EA_TRY(ensure_regions(t, dir, n));
  DirRes &R = t->res[dir];
  const int r = R.next;
  R.next = (R.next + 1) % kRegions;
  if (R.used[r]) EA_HIP(hipEventSynchronize(R.ev[r]));
  if (slots) std::memcpy(R.h[r], slots, (size_t)n * 8);
  std::memcpy(R.h[r] + n * 8, pages, (size_t)n * 4);
  EA_HIP(hipMemcpyAsync(R.d[r], R.h[r], (size_t)n * 12, hipMemcpyHostToDevice, s));
  *d_slots = reinterpret_cast<const int64_t *>(R.d[r]);
  *d_pages = reinterpret_cast<const int32_t *>(R.d[r] + n * 8);
  *region = r;
  return EA_OK;
}

int release_region(ea_tier *t, int dir, int r, hipStream_t s) {
  DirRes &R = t->res[dir];
  EA_HIP(hipEventRecord(R.ev[r], s));
  R.used[r] = true;
  return EA_OK;
}

int ensure_staging(ea_tier *t, int dir) {
  DirRes &R = t->res[dir];
  if (R.staging) return EA_OK;
  int64_t half = default_staging_bytes() / 2;
  int64_t per_half = std::max<int64_t>(1, half / t->slot);
  EA_HIP(hipMalloc((void **)&R.staging, (size_t)(2 * per_half * t->slot)));
  EA_HIP(hipEventCreateWithFlags(&R.staging_ev, hipEventDisableTiming));
  R.per_half = per_half;
  return EA_OK;
}

int32_t new_event(ea_tier *t, hipStream_t s) {
  int32_t e;
  if (!t->free_evs.empty()) {
    e = t->free_evs.back();
    t->free_evs.pop_back();
  } else {
    hipEvent_t ev;
    if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) return -1;
    t->evs.push_back(EvRec{ev, nullptr, 0});
    e = (int32_t)t->evs.size() - 1;
  }
  t->evs[e].stream = s;
  t->evs[e].refs = 0;
  return e;
}

void unref_event(ea_tier *t, int32_t e) {
  if (e < 0) return;
  if (--t->evs[e].refs == 0) t->free_evs.push_back(e);
}

// Order `s` after earlier transfers on other streams that touch these slots.
int wait_slot_hazards(ea_tier *t, const int64_t *slots, const uint8_t *mask,
                      int64_t n, hipStream_t s) {
  std::vector<int32_t> waits;
  for (int64_t i = 0; i < n; ++i) {
    if (mask && !mask[i]) continue;
    const int32_t e = t->slot_ev[slots[i]];
    if (e < 0 || t->evs[e].stream == s) continue;
    if (std::find(waits.begin(), waits.end(), e) == waits.end()) waits.push_back(e);
  }
  for (int32_t e : waits) {
    hipError_t q = hipEventQuery(t->evs[e].ev);
    if (q == hipSuccess) continue;
    if (q != hipErrorNotReady) {
      g_last_hip = (int)q;
      return EA_EHIP;
    }
    EA_HIP(hipStreamWaitEvent(s, t->evs[e].ev, 0));
  }
  return EA_OK;
}

// Record the end of this call's transfer on `s` as the slots' last event.
int note_slot_transfer(ea_tier *t, const int64_t *slots, const uint8_t *mask,
                       int64_t n, hipStream_t s) {
  const int32_t e = new_event(t, s);
  if (e < 0) {
    g_last_hip = (int)hipErrorOutOfMemory;
    return EA_EHIP;
  }
  EA_HIP(hipEventRecord(t->evs[e].ev, s));
  for (int64_t i = 0; i < n; ++i) {
    if (mask && !mask[i]) continue;
    int32_t &cur = t->slot_ev[slots[i]];
    if (cur == e) continue;
    unref_event(t, cur);
    cur = e;
    t->evs[e].refs += 1;
  }
  if (t->evs[e].refs == 0) t->free_evs.push_back(e);
  return EA_OK;
}

bool same_shape(const ea_tier *t, const ea_cache *c) {
  return c->d.num_layers == t->num_layers && c->piece == t->piece &&
         (c->d.scale_base != nullptr) == (t->has_scales != 0);
}

ea::PieceCopy base_copy(const ea_cache *c, int64_t slot_bytes) {
  ea::PieceCopy a{};
  a.cache = static_cast<uint8_t *>(c->d.base);
  a.scales = static_cast<uint8_t *>(c->d.scale_base);
  a.num_pages = c->d.num_pages;
  a.piece_bytes = c->piece;
  a.slot_bytes = slot_bytes;
  a.page_bytes = c->page;
  a.num_layers = c->d.num_layers;
  a.layer_begin = 0;
  a.layer_count = c->d.num_layers;
  return a;
}

// Direct plan: one kernel between the cache and the mapped pinned slots.
int copy_direct(ea_tier *t, ea_cache *c, const int64_t *slots,
                const int32_t *pages, int64_t n, int dir, int layer_begin,
                int layer_count, hipStream_t s, int res_dir) {
  ea::PieceCopy a = base_copy(c, t->slot);
  a.slots = t->dev;
  a.n = n;
  a.layer_begin = layer_begin;
  a.layer_count = layer_count;
  if (n <= ea::kInlineMax) {
    ea::InlineIdx inl;
    for (int64_t i = 0; i < n; ++i) {
      inl.pages[i] = pages[i];
      inl.slots[i] = slots[i];
    }
    EA_HIP(ea::launch_piece_copy(a, &inl, dir, t->grid_cap, s));
    return EA_OK;
  }
  int region;
  EA_TRY(upload_indices(t, res_dir, slots, pages, n, s, &a.slot_idx, &a.pages, &region));
  EA_HIP(ea::launch_piece_copy(a, nullptr, dir, t->grid_cap, s));
  return release_region(t, res_dir, region, s);
}

// Staged plan: HBM staging + DMA copies of runs of consecutive slots.
// Entries are processed in slot order so that consecutive slots coalesce.
int copy_staged(ea_tier *t, ea_cache *c, const int64_t *slots,
                const int32_t *pages, int64_t n, int dir, hipStream_t s) {
  const int res_dir = dir == ea::kToSlots ? EA_DIR_STORE : EA_DIR_LOAD;
  EA_TRY(ensure_staging(t, res_dir));
  DirRes &R = t->res[res_dir];
  if (R.staging_used && R.staging_stream != s) EA_HIP(hipStreamWaitEvent(s, R.staging_ev, 0));

  std::vector<int64_t> order((size_t)n);
  for (int64_t i = 0; i < n; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(),
                   [&](int64_t x, int64_t y) { return slots[x] < slots[y]; });
  std::vector<int64_t> ss((size_t)n);
  std::vector<int32_t> pp((size_t)n);
  for (int64_t i = 0; i < n; ++i) {
    ss[i] = slots[order[i]];
    pp[i] = pages[order[i]];
  }
  const int64_t *d_slots;
  const int32_t *d_pages;
  int region;
  EA_TRY(upload_indices(t, res_dir, nullptr, pp.data(), n, s, &d_slots, &d_pages, &region));

  const int64_t per = R.per_half;
  for (int64_t c0 = 0, chunk = 0; c0 < n; c0 += per, ++chunk) {
    const int64_t c1 = std::min(n, c0 + per);
    uint8_t *stage = R.staging + (chunk & 1) * per * t->slot;
    ea::PieceCopy a = base_copy(c, t->slot);
    a.slots = stage;
    a.pages = d_pages + c0;
    a.identity_slots = 1;
    a.n = c1 - c0;
    if (dir == ea::kToSlots) EA_HIP(ea::launch_piece_copy(a, nullptr, dir, t->grid_cap, s));
    for (int64_t j0 = c0; j0 < c1;) {
      int64_t j1 = j0 + 1;
      while (j1 < c1 && ss[j1] == ss[j1 - 1] + 1) ++j1;
      uint8_t *h = t->host + ss[j0] * t->slot;
      uint8_t *g = stage + (j0 - c0) * t->slot;
      const size_t bytes = (size_t)((j1 - j0) * t->slot);
      if (dir == ea::kToSlots)
        EA_HIP(hipMemcpyAsync(h, g, bytes, hipMemcpyDeviceToHost, s));
      else
        EA_HIP(hipMemcpyAsync(g, h, bytes, hipMemcpyHostToDevice, s));
      j0 = j1;
    }
    if (dir == ea::kToPages) EA_HIP(ea::launch_piece_copy(a, nullptr, dir, t->grid_cap, s));
  }
  EA_TRY(release_region(t, res_dir, region, s));
  EA_HIP(hipEventRecord(R.staging_ev, s));
  R.staging_used = true;
  R.staging_stream = s;
  return EA_OK;
}

int validate_cache_desc(const ea_cache_desc *d) {
  if (!d || !d->base) return EA_EINVAL;
  if (d->num_pages < 1 || d->num_layers < 1 || d->page_tokens < 1 ||
      d->num_kv_heads < 1 || d->head_dim < 1 || d->elem_bytes < 1)
    return EA_EINVAL;
  const int64_t piece = 2LL * d->page_tokens * d->num_kv_heads * d->head_dim * d->elem_bytes;
  if (piece % 16 != 0) return EA_EINVAL;
  if (!aligned(d->base, 16)) return EA_EINVAL;
  if (d->scale_base && !aligned(d->scale_base, 8)) return EA_EINVAL;
  return EA_OK;
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
  c->piece = 2LL * desc->page_tokens * desc->num_kv_heads * desc->head_dim * desc->elem_bytes;
  c->page = c->piece * desc->num_layers;
  c->trailer = desc->scale_base ? ((int64_t)desc->num_layers * 8 + 255) / 256 * 256 : 0;
  c->slot = c->page + c->trailer;
  *out = c;
  return EA_OK;
}

int ea_cache_destroy(ea_cache *cache) {
  if (!cache) return EA_EINVAL;
  delete cache;
  return EA_OK;
}

int ea_tier_create(const ea_cache *shape, int64_t capacity_bytes, int numa_node,
                   ea_tier **out) {
  if (!shape || !out || capacity_bytes <= 0) return EA_EINVAL;
  const int64_t K = capacity_bytes / shape->slot;
  if (K < 1) return EA_EINVAL;
  DeviceScope ds(shape->device);
  EA_TRY(ds.status());
  std::unique_ptr<ea_tier> t(new (std::nothrow) ea_tier);
  if (!t) return EA_ENOMEM;
  t->device = shape->device;
  t->num_layers = shape->d.num_layers;
  t->has_scales = shape->d.scale_base != nullptr;
  t->piece = shape->piece;
  t->page = shape->page;
  t->trailer = shape->trailer;
  t->slot = shape->slot;
  t->K = K;
  t->capacity_bytes = capacity_bytes;
  t->grid_cap = env_int("EA_GRID", 0);
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
  hipError_t e = hipHostMalloc((void **)&t->host, (size_t)(K * t->slot), flags);
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
  t->meta.reset(new (std::nothrow) ea::TierMeta(K, capacity_bytes));
  if (!t->meta) {
    (void)hipHostFree(t->host);
    return EA_ENOMEM;
  }
  t->slot_ev.assign((size_t)K, -1);
  *out = t.release();
  return EA_OK;
}

int ea_tier_destroy(ea_tier *t) {
  if (!t) return EA_EINVAL;
  {
    DeviceScope ds(t->device);
    std::lock_guard<std::mutex> lk(t->mu);
    for (auto &ev : t->evs) {
      (void)hipEventSynchronize(ev.ev);
      (void)hipEventDestroy(ev.ev);
    }
    for (auto &R : t->res) {
      for (int r = 0; r < kRegions; ++r) {
        if (R.ev[r]) {
          (void)hipEventSynchronize(R.ev[r]);
          (void)hipEventDestroy(R.ev[r]);
        }
        if (R.h[r]) (void)hipHostFree(R.h[r]);
        if (R.d[r]) (void)hipFree(R.d[r]);
      }
      if (R.staging_ev) {
        (void)hipEventSynchronize(R.staging_ev);
        (void)hipEventDestroy(R.staging_ev);
      }
      if (R.staging) (void)hipFree(R.staging);
    }
    if (t->host) (void)hipHostFree(t->host);
  }
  delete t;
  return EA_OK;
}

int ea_tier_get_info(const ea_tier *t, ea_tier_info *info) {
  if (!t || !info) return EA_EINVAL;
  info->capacity_slots = t->K;
  info->slot_bytes = t->slot;
  info->piece_bytes = t->piece;
  info->page_bytes = t->page;
  info->trailer_bytes = t->trailer;
  info->capacity_bytes = t->capacity_bytes;
  info->host_base = t->host;
  info->device_base = t->dev;
  return EA_OK;
}

int ea_tier_lookup(ea_tier *t, const uint8_t *keys, int64_t n, int64_t *hit_blocks,
                   int64_t *slots_out) {
  if (!t || n < 0 || !hit_blocks) return EA_EINVAL;
  if (n > 0 && (!keys || !slots_out)) return EA_EINVAL;
  std::lock_guard<std::mutex> lk(t->mu);
  return t->meta->lookup(keys, n, hit_blocks, slots_out);
}

int ea_admission_fill(ea_tier *t, const ea_policy *p, const ea_request *r,
                      const uint8_t *keys, int64_t n_keys, uint8_t *mask_out,
                      int32_t *save_out) {
  if (!t || !p || !r || !save_out || n_keys < 0) return EA_EINVAL;
  if (n_keys > 0 && (!keys || !mask_out)) return EA_EINVAL;
  std::lock_guard<std::mutex> lk(t->mu);
  return t->meta->admission(*p, *r, keys, n_keys, mask_out, save_out);
}

int ea_tier_alloc(ea_tier *t, const uint8_t *keys, const uint8_t *mask, int64_t n,
                  int64_t *slots_out, int64_t *allocated) {
  if (!t || n < 0 || !allocated) return EA_EINVAL;
  if (n > 0 && (!keys || !slots_out)) return EA_EINVAL;
  std::lock_guard<std::mutex> lk(t->mu);
  return t->meta->alloc(keys, mask, n, slots_out, allocated);
}

int ea_tier_unpin(ea_tier *t, const int64_t *slots, int64_t n) {
  if (!t || n < 0) return EA_EINVAL;
  if (n == 0) return EA_OK;
  if (!slots) return EA_EINVAL;
  std::lock_guard<std::mutex> lk(t->mu);
  return t->meta->unpin(slots, n);
}

int ea_tier_stats_get(const ea_tier *t, ea_tier_stats *s) {
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
  if (!c || !t || n < 0) return EA_EINVAL;
  if (!same_shape(t, c)) return EA_EINVAL;
  if (n == 0) return EA_OK;
  if (!block_ids || !host_slots) return EA_EINVAL;
  std::vector<int64_t> slots;
  std::vector<int32_t> pages;
  slots.reserve((size_t)n);
  pages.reserve((size_t)n);
  for (int32_t i = 0; i < n; ++i) {
    if (admit_mask && !admit_mask[i]) continue;
    if (block_ids[i] < 0 || block_ids[i] >= c->d.num_pages) return EA_EINVAL;
    if (host_slots[i] < 0 || host_slots[i] >= t->K) return EA_EINVAL;
    slots.push_back(host_slots[i]);
    pages.push_back(block_ids[i]);
  }
  if (!all_distinct(slots.data(), (int64_t)slots.size())) return EA_EINVAL;
  const int64_t m = (int64_t)slots.size();
  if (m == 0) return EA_OK;
  DeviceScope ds(t->device);
  EA_TRY(ds.status());
  std::lock_guard<std::mutex> lk(t->mu);
  EA_TRY(wait_slot_hazards(t, slots.data(), nullptr, m, stream));
  if (resolve_plan(t, EA_DIR_STORE) == EA_PLAN_STAGED)
    EA_TRY(copy_staged(t, c, slots.data(), pages.data(), m, ea::kToSlots, stream));
  else
    EA_TRY(copy_direct(t, c, slots.data(), pages.data(), m, ea::kToSlots, 0,
                       c->d.num_layers, stream, EA_DIR_STORE));
  EA_TRY(note_slot_transfer(t, slots.data(), nullptr, m, stream));
  for (int64_t i = 0; i < m; ++i) t->meta->mark_stored(slots[i]);
  t->bytes_stored += m * t->slot;
  t->store_calls += 1;
  return EA_OK;
}

static int validate_load(ea_tier *t, ea_cache *c, const int64_t *host_slots,
                         const int32_t *dst_pages, int32_t n) {
  if (!c || !t || n < 0) return EA_EINVAL;
  if (!same_shape(t, c)) return EA_EINVAL;
  if (n == 0) return EA_OK;
  if (!host_slots || !dst_pages) return EA_EINVAL;
  for (int32_t i = 0; i < n; ++i) {
    if (dst_pages[i] < 0 || dst_pages[i] >= c->d.num_pages) return EA_EINVAL;
    if (host_slots[i] < 0 || host_slots[i] >= t->K) return EA_EINVAL;
  }
  if (!all_distinct(dst_pages, n)) return EA_EINVAL;
  return EA_OK;
}

int ea_load_blocks(ea_tier *t, ea_cache *c, const int64_t *host_slots,
                   const int32_t *dst_pages, int32_t n, hipStream_t stream) {
  EA_TRY(validate_load(t, c, host_slots, dst_pages, n));
  if (n == 0) return EA_OK;
  DeviceScope ds(t->device);
  EA_TRY(ds.status());
  std::lock_guard<std::mutex> lk(t->mu);
  EA_TRY(wait_slot_hazards(t, host_slots, nullptr, n, stream));
  if (resolve_plan(t, EA_DIR_LOAD) == EA_PLAN_STAGED)
    EA_TRY(copy_staged(t, c, host_slots, dst_pages, n, ea::kToPages, stream));
  else
    EA_TRY(copy_direct(t, c, host_slots, dst_pages, n, ea::kToPages, 0,
                       c->d.num_layers, stream, EA_DIR_LOAD));
  EA_TRY(note_slot_transfer(t, host_slots, nullptr, n, stream));
  t->bytes_loaded += (int64_t)n * t->slot;
  t->load_calls += 1;
  return EA_OK;
}

int ea_load_blocks_layered(ea_tier *t, ea_cache *c, const int64_t *host_slots,
                           const int32_t *dst_pages, int32_t n,
                           hipStream_t copy_stream, hipEvent_t *layer_done) {
  if (!layer_done) return EA_EINVAL;
  EA_TRY(validate_load(t, c, host_slots, dst_pages, n));
  for (int32_t l = 0; l < (c ? c->d.num_layers : 0); ++l)
    if (!layer_done[l]) return EA_EINVAL;
  DeviceScope ds(t->device);
  EA_TRY(ds.status());
  std::lock_guard<std::mutex> lk(t->mu);
  if (n == 0) {
    for (int32_t l = 0; l < c->d.num_layers; ++l)
      EA_HIP(hipEventRecord(layer_done[l], copy_stream));
    return EA_OK;
  }
  EA_TRY(wait_slot_hazards(t, host_slots, nullptr, n, copy_stream));
  // the pieces of one layer are strided inside the slots, so every layer is
  // its own direct kernel over all n slots
  ea::PieceCopy a = base_copy(c, t->slot);
  a.slots = t->dev;
  a.n = n;
  a.layer_count = 1;
  ea::InlineIdx inl;
  const ea::InlineIdx *pin = nullptr;
  int region = -1;
  if (n <= ea::kInlineMax) {
    for (int32_t i = 0; i < n; ++i) {
      inl.pages[i] = dst_pages[i];
      inl.slots[i] = host_slots[i];
    }
    pin = &inl;
  } else {
    EA_TRY(upload_indices(t, EA_DIR_LOAD, host_slots, dst_pages, n, copy_stream,
                          &a.slot_idx, &a.pages, &region));
  }
  for (int32_t l = 0; l < c->d.num_layers; ++l) {
    a.layer_begin = l;
    EA_HIP(ea::launch_piece_copy(a, pin, ea::kToPages, t->grid_cap, copy_stream));
    EA_HIP(hipEventRecord(layer_done[l], copy_stream));
  }
  if (region >= 0) EA_TRY(release_region(t, EA_DIR_LOAD, region, copy_stream));
  EA_TRY(note_slot_transfer(t, host_slots, nullptr, n, copy_stream));
  t->bytes_loaded += (int64_t)n * t->slot;
  t->load_calls += 1;
  return EA_OK;
}

// ------------------------------------------------- gather / scatter (HBM)

namespace {

struct GatherWs {
  std::mutex mu;
  int32_t *h = nullptr;
  int32_t *d = nullptr;
  int64_t cap = 0;
  hipEvent_t ev = nullptr;
  bool used = false;
};
GatherWs g_gather;

int gather_scatter(ea_cache *c, const int32_t *pages, int32_t n, void *buf,
                   int dir, hipStream_t s) {
  const int64_t slot = c->slot;
  DeviceScope ds(c->device);
  EA_TRY(ds.status());
  ea::PieceCopy a = base_copy(c, slot);
  a.slots = static_cast<uint8_t *>(buf);
  a.n = n;
  a.identity_slots = 1;
  if (n <= ea::kInlineMax) {
    ea::InlineIdx inl;
    for (int32_t i = 0; i < n; ++i) {
      inl.pages[i] = pages[i];
      inl.slots[i] = i;
    }
    EA_HIP(ea::launch_piece_copy(a, &inl, dir, env_int("EA_GRID", 0), s));
    return EA_OK;
  }
  std::lock_guard<std::mutex> lk(g_gather.mu);
  if (g_gather.used) EA_HIP(hipEventSynchronize(g_gather.ev));
  if (n > g_gather.cap) {
    if (g_gather.h) (void)hipHostFree(g_gather.h);
    if (g_gather.d) (void)hipFree(g_gather.d);
    g_gather.h = nullptr;
    g_gather.d = nullptr;
    g_gather.cap = 0;
    const int64_t cap = std::max<int64_t>(n, 4096);
    EA_HIP(hipHostMalloc((void **)&g_gather.h, (size_t)cap * 4, hipHostMallocDefault));
    EA_HIP(hipMalloc((void **)&g_gather.d, (size_t)cap * 4));
    g_gather.cap = cap;
  }
  if (!g_gather.ev) EA_HIP(hipEventCreateWithFlags(&g_gather.ev, hipEventDisableTiming));
  std::memcpy(g_gather.h, pages, (size_t)n * 4);
  EA_HIP(hipMemcpyAsync(g_gather.d, g_gather.h, (size_t)n * 4, hipMemcpyHostToDevice, s));
  a.pages = g_gather.d;
  EA_HIP(ea::launch_piece_copy(a, nullptr, dir, env_int("EA_GRID", 0), s));
  EA_HIP(hipEventRecord(g_gather.ev, s));
  g_gather.used = true;
  return EA_OK;
}

}  // namespace

int ea_gather_blocks(ea_cache *c, const int32_t *block_ids, int32_t n, void *d_dst,
                     hipStream_t stream) {
  if (!c || n < 0) return EA_EINVAL;
  if (n == 0) return EA_OK;
  if (!block_ids || !d_dst || !aligned(d_dst, 16)) return EA_EINVAL;
  for (int32_t i = 0; i < n; ++i)
    if (block_ids[i] < 0 || block_ids[i] >= c->d.num_pages) return EA_EINVAL;
  return gather_scatter(c, block_ids, n, d_dst, ea::kToSlots, stream);
}

int ea_scatter_blocks(ea_cache *c, const void *d_src, const int32_t *dst_pages,
                      int32_t n, hipStream_t stream) {
  if (!c || n < 0) return EA_EINVAL;
  if (n == 0) return EA_OK;
  if (!dst_pages || !d_src || !aligned(d_src, 16)) return EA_EINVAL;
  for (int32_t i = 0; i < n; ++i)
    if (dst_pages[i] < 0 || dst_pages[i] >= c->d.num_pages) return EA_EINVAL;
  if (!all_distinct(dst_pages, n)) return EA_EINVAL;
  return gather_scatter(c, dst_pages, n, const_cast<void *>(d_src), ea::kToPages, stream);
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
  for (auto &ev : t->evs) EA_HIP(hipEventSynchronize(ev.ev));
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
  for (int r = 0; r < reps && rc == EA_OK; ++r) {
    hipError_t e = hipSuccess;
    const int streams = direction == EA_DIR_BOTH ? 2 : 1;
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
    const double g = (double)(streams * bytes) / (worst * 1e-3) / 1e9;
    best = std::max(best, g);
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
