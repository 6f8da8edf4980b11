// Hash entry points of libea: chained prefix-block keys on the GPU.
//
// Buffers live in one workspace per (device, stream).  A call locks only its
// own workspace, so threads hashing on different streams never wait for one
// another; calls on one stream are ordered by the stream anyway.  Workspaces
// are grow-only and kept until the process ends.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <climits>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <memory>
#include <mutex>
#include <vector>

#include "ea.h"
#include "ea_internal.hpp"

namespace {

#define HS_HIP(expr)               \
  do {                             \
    hipError_t e_ = (expr);        \
    if (e_ != hipSuccess) {        \
      ea::set_last_hip((int)e_);   \
      return EA_EHIP;              \
    }                              \
  } while (0)

// Offsets and midstates of one asynchronous (device) call with host
// offsets.  Two of them alternate, so the host prepares the next call while
// the GPU runs one.
struct DevSlot {
  uint8_t *h_meta = nullptr, *d_meta = nullptr;
  int64_t cap_meta = 0;
  uint32_t *d_mid = nullptr;
  int64_t cap_mid = 0;  // keys
  hipEvent_t done = nullptr;
  bool used = false;
};

// Grow-only device/pinned buffers of the calls on one stream of one device.
struct HashWs {
  int device = -1;
  hipStream_t stream = nullptr;
  std::mutex mu;  // one call at a time on this workspace
  // End of a call's use of the buffers.  `done` ends a call whose results
  // the host reads (its record carries the system-scope release that makes
  // them visible there); `done_dev` ends a call whose results stay on the
  // device, and skips that release (it only orders later work and buffer
  // reuse).  `last` is whichever event the last call recorded.
  hipEvent_t done = nullptr;
  hipEvent_t done_dev = nullptr;
  hipEvent_t last = nullptr;
  bool used = false;
  // ea_hash_blocks: pinned host staging
  uint8_t *h_tok = nullptr;  int64_t cap_tok = 0;   // bytes
  uint8_t *h_meta = nullptr; int64_t cap_meta = 0;  // offsets + parents
  uint8_t *h_keys = nullptr; int64_t cap_keys = 0;  // bytes
  uint8_t *d_tok = nullptr;
  uint8_t *d_meta = nullptr;
  uint8_t *d_keys = nullptr;
  uint32_t *d_mid = nullptr; int64_t cap_mid = 0;   // keys
  DevSlot slots[2];                                 // ea_hash_blocks_device
  int next = 0;
  // ea_hash_blocks_device_offsets: offsets derived on the device, and the
  // scan's state (its first 8 bytes, a ticket counter, zero between calls)
  uint8_t *d_off = nullptr;  int64_t cap_off = 0;   // bytes
  uint8_t *d_scan = nullptr; int64_t cap_scan = 0;  // bytes
};

std::mutex g_ws_mu;  // guards the list only, never held across a HIP wait
std::vector<std::unique_ptr<HashWs>> g_ws;

// The workspace of (current device, stream), created on first use.
int workspace(hipStream_t stream, HashWs **out) {
  int dev;
  HS_HIP(hipGetDevice(&dev));
  std::lock_guard<std::mutex> lk(g_ws_mu);
  for (auto &w : g_ws)
    if (w->device == dev && w->stream == stream) {
      *out = w.get();
      return EA_OK;
    }
  std::unique_ptr<HashWs> w(new (std::nothrow) HashWs);
  if (!w) return EA_ENOMEM;
  w->device = dev;
  w->stream = stream;
  HS_HIP(hipEventCreateWithFlags(&w->done, hipEventDisableTiming));
  HS_HIP(hipEventCreateWithFlags(&w->done_dev, ea::kDeviceEventFlags));
  *out = w.get();
  g_ws.push_back(std::move(w));
  return EA_OK;
}

// Order the stream after the workspace's last use.  Calls on one stream are
// ordered already; this covers a stream handle that a destroyed stream's
// successor reuses.
int after_last_use(HashWs &w, hipStream_t stream) {
  if (w.used) HS_HIP(hipStreamWaitEvent(stream, w.last, 0));
  return EA_OK;
}

// Mark the end of this call's use of the buffers on `stream`; host_reads:
// the host reads what the call wrote once the event has fired.
int release(HashWs &w, hipStream_t stream, bool host_reads) {
  hipEvent_t e = host_reads ? w.done : w.done_dev;
  HS_HIP(hipEventRecord(e, stream));
  w.last = e;
  w.used = true;
  return EA_OK;
}

// Grow a pinned host buffer (and its device twin when d is not null).  The
// old buffers may still be read by the stream's earlier work: wait for it.
int grow_pair(HashWs &w, uint8_t **h, uint8_t **d, int64_t *cap, int64_t need) {
  if (need <= *cap) return EA_OK;
  if (w.used) HS_HIP(hipEventSynchronize(w.last));
  if (*h) (void)hipHostFree(*h);
  if (d && *d) (void)hipFree(*d);
  *h = nullptr;
  if (d) *d = nullptr;
  *cap = 0;
  const int64_t c = std::max<int64_t>(need, 1 << 16);
  HS_HIP(hipHostMalloc((void **)h, (size_t)c, hipHostMallocDefault));
  if (d) HS_HIP(hipMalloc((void **)d, (size_t)c));
  *cap = c;
  return EA_OK;
}

int grow_device(HashWs &w, uint8_t **d, int64_t *cap, int64_t need) {
  if (need <= *cap) return EA_OK;
  if (w.used) HS_HIP(hipEventSynchronize(w.last));
  if (*d) (void)hipFree(*d);
  *d = nullptr;
  *cap = 0;
  const int64_t c = std::max<int64_t>(need, 1 << 16);
  HS_HIP(hipMalloc((void **)d, (size_t)c));
  *cap = c;
  return EA_OK;
}

int ensure_mid(HashWs &w, uint32_t **mid, int64_t *cap, int64_t keys) {
  if (keys <= *cap) return EA_OK;
  if (w.used) HS_HIP(hipEventSynchronize(w.last));
  if (*mid) (void)hipFree(*mid);
  *mid = nullptr;
  *cap = 0;
  const int64_t c = std::max<int64_t>(keys, 4096);
  HS_HIP(hipMalloc((void **)mid, (size_t)c * 32));
  *cap = c;
  return EA_OK;
}

// floor(len / b), the full blocks of a sequence: a shift when b is a power
// of two (16-token pages, 1,024-token chunks), else a division.
struct BlockCount {
  int64_t b;
  int shift = -1;
  explicit BlockCount(int64_t block) : b(block) {
    if ((b & (b - 1)) == 0) shift = __builtin_ctzll((unsigned long long)b);
  }
  int64_t operator()(int64_t len) const { return shift >= 0 ? len >> shift : len / b; }
};

int check_block(int32_t block_tokens) {
  if (block_tokens < 1 || block_tokens > (1 << 20)) return EA_EINVAL;
  if (block_tokens % 16 != 0) return EA_ENOTSUP;
  return EA_OK;
}

// Checks host sequence offsets against the n_tokens tokens given and fills
// key_offsets_out (running sums of full blocks) in one pass.
int validate(const int64_t *seq_offsets, int32_t n_seqs, int64_t n_tokens, int32_t block_tokens,
             int64_t *key_offsets_out, int64_t *total_keys) {
  if (n_seqs < 0 || !key_offsets_out || !seq_offsets) return EA_EINVAL;
  const int rc = check_block(block_tokens);
  if (rc != EA_OK) return rc;
  const BlockCount blocks(block_tokens);
  int64_t k = 0;
  key_offsets_out[0] = 0;
  if (seq_offsets[0] < 0 || seq_offsets[0] > n_tokens) return EA_EINVAL;
  for (int32_t s = 0; s < n_seqs; ++s) {
    const int64_t a = seq_offsets[s], e = seq_offsets[s + 1];
    if (e < a || e > n_tokens) return EA_EINVAL;
    k += blocks(e - a);
    key_offsets_out[s + 1] = k;
  }
  *total_keys = k;
  return EA_OK;
}

// Key offsets [n+1] then token offsets [n] for the kernels, written at h as
// int32 when `wide` is false (every value below 2^31: half the bytes to
// upload) and int64 otherwise.  Token offsets are toff[s], or koff[s] * b
// for tokens packed block after block (toff null).
template <typename Off>
void write_offsets(uint8_t *h, const int64_t *koff, const int64_t *toff, int64_t b,
                   int32_t n) {
  Off *k = reinterpret_cast<Off *>(h);
  Off *t = k + n + 1;
  for (int32_t s = 0; s <= n; ++s) k[s] = (Off)koff[s];
  if (toff)
    for (int32_t s = 0; s < n; ++s) t[s] = (Off)toff[s];
  else
    for (int32_t s = 0; s < n; ++s) t[s] = (Off)(koff[s] * b);
}

// EA_HASH_OFFSETS=64 keeps 64-bit offsets even where 32 bits would do.
bool force_wide() {
  const char *v = std::getenv("EA_HASH_OFFSETS");
  return v && std::strcmp(v, "64") == 0;
}

// Bytes of the kernels' offsets, rounded up to 16.
int64_t offsets_bytes(int32_t n, bool wide) {
  return ((2 * (int64_t)n + 1) * (wide ? 8 : 4) + 15) / 16 * 16;
}

void put_offsets(uint8_t *h, const int64_t *koff, const int64_t *toff, int64_t b, int32_t n,
                 bool wide) {
  if (wide)
    write_offsets<int64_t>(h, koff, toff, b, n);
  else
    write_offsets<int32_t>(h, koff, toff, b, n);
}

// The hash kernels after the offsets are in place on the device.
int run_kernels(const int32_t *d_tokens, const uint8_t *d_koff, const uint8_t *d_toff, bool wide,
                int32_t n_seqs, int64_t key_bound, int32_t block_tokens, uint32_t *d_mid,
                const uint8_t *d_parents, uint8_t *d_keys, hipStream_t stream) {
  if (ea::hash_fused(n_seqs)) {
    HS_HIP(ea::launch_sha256_fused(d_tokens, d_koff, d_toff, wide, n_seqs, block_tokens,
                                   d_parents, d_keys, stream));
    return EA_OK;
  }
  HS_HIP(ea::launch_sha256_midstates(d_tokens, d_koff, d_toff, wide, n_seqs, key_bound,
                                     block_tokens, d_mid, stream));
  HS_HIP(ea::launch_sha256_chain(d_mid, d_koff, wide, n_seqs, block_tokens, d_parents, d_keys,
                                 stream));
  return EA_OK;
}

}  // namespace

extern "C" int ea_hash_blocks(const int32_t *tokens, const int64_t *seq_offsets,
                              int32_t n_seqs, int32_t block_tokens,
                              const uint8_t *parents, uint8_t *keys_out,
                              int64_t *key_offsets_out, hipStream_t stream) {
  int64_t total = 0;
  if (!seq_offsets) return EA_EINVAL;
  // the tokens array is as long as the last sequence's end
  int rc = validate(seq_offsets, n_seqs, n_seqs >= 0 ? seq_offsets[n_seqs] : 0, block_tokens,
                    key_offsets_out, &total);
  if (rc != EA_OK) return rc;
  if (total > 0 && (!tokens || !keys_out)) return EA_EINVAL;
  if (total == 0) return EA_OK;

  HashWs *wp = nullptr;
  if ((rc = workspace(stream, &wp)) != EA_OK) return rc;
  HashWs &w = *wp;
  std::lock_guard<std::mutex> lk(w.mu);
  // the previous call on this stream has returned its keys already, but a
  // reused stream handle may not be ordered after it
  if (w.used) HS_HIP(hipEventSynchronize(w.last));
  // pack the full-block tokens of every sequence contiguously
  const int64_t tok_bytes = total * block_tokens * 4;
  const bool wide = total * block_tokens > INT32_MAX || force_wide();
  const int64_t off_bytes = offsets_bytes(n_seqs, wide);
  const int64_t meta_bytes = off_bytes + (parents ? 32 * (int64_t)n_seqs : 0);
  if ((rc = grow_pair(w, &w.h_tok, &w.d_tok, &w.cap_tok, tok_bytes)) != EA_OK) return rc;
  if ((rc = grow_pair(w, &w.h_meta, &w.d_meta, &w.cap_meta, meta_bytes)) != EA_OK) return rc;
  if ((rc = grow_pair(w, &w.h_keys, &w.d_keys, &w.cap_keys, total * 32)) != EA_OK) return rc;
  if ((rc = ensure_mid(w, &w.d_mid, &w.cap_mid, total)) != EA_OK) return rc;

  for (int32_t s = 0; s < n_seqs; ++s) {
    const int64_t nt = (key_offsets_out[s + 1] - key_offsets_out[s]) * block_tokens;
    std::memcpy(w.h_tok + key_offsets_out[s] * block_tokens * 4, tokens + seq_offsets[s],
                (size_t)nt * 4);
  }
  put_offsets(w.h_meta, key_offsets_out, nullptr, block_tokens, n_seqs, wide);
  if (parents) std::memcpy(w.h_meta + off_bytes, parents, (size_t)n_seqs * 32);

  HS_HIP(hipMemcpyAsync(w.d_tok, w.h_tok, (size_t)tok_bytes, hipMemcpyHostToDevice, stream));
  HS_HIP(hipMemcpyAsync(w.d_meta, w.h_meta, (size_t)meta_bytes, hipMemcpyHostToDevice, stream));
  const uint8_t *d_koff = w.d_meta;
  const uint8_t *d_toff = d_koff + (n_seqs + 1) * (wide ? 8 : 4);
  const uint8_t *d_par = parents ? w.d_meta + off_bytes : nullptr;
  if ((rc = run_kernels(reinterpret_cast<const int32_t *>(w.d_tok), d_koff, d_toff, wide,
                        n_seqs, total, block_tokens, w.d_mid, d_par, w.d_keys, stream)) != EA_OK)
    return rc;
  HS_HIP(hipMemcpyAsync(w.h_keys, w.d_keys, (size_t)total * 32, hipMemcpyDeviceToHost, stream));
  if ((rc = release(w, stream, true)) != EA_OK) return rc;
  HS_HIP(hipEventSynchronize(w.done));  // this workspace's lock only
  std::memcpy(keys_out, w.h_keys, (size_t)total * 32);
  return EA_OK;
}

extern "C" int ea_hash_blocks_device(const int32_t *d_tokens, int64_t n_tokens,
                                     const int64_t *seq_offsets, int32_t n_seqs,
                                     int32_t block_tokens, const uint8_t *d_parents,
                                     uint8_t *d_keys_out, int64_t keys_capacity,
                                     int64_t *key_offsets_out, hipStream_t stream) {
  int64_t total = 0;
  if (n_tokens < 0 || keys_capacity < 0) return EA_EINVAL;
  int rc = validate(seq_offsets, n_seqs, n_tokens, block_tokens, key_offsets_out, &total);
  if (rc != EA_OK) return rc;
  if (total > keys_capacity) return EA_EINVAL;
  if (total > 0 && (!d_tokens || !d_keys_out)) return EA_EINVAL;
  if (d_keys_out && ((uintptr_t)d_keys_out & 15) != 0) return EA_EINVAL;
  if (total == 0) return EA_OK;

  HashWs *wp = nullptr;
  if ((rc = workspace(stream, &wp)) != EA_OK) return rc;
  HashWs &w = *wp;
  std::lock_guard<std::mutex> lk(w.mu);
  DevSlot &d = w.slots[w.next];
  w.next ^= 1;
  // the call two back on this stream still reads this slot's host offsets
  if (d.used) HS_HIP(hipEventSynchronize(d.done));
  if (!d.done) HS_HIP(hipEventCreateWithFlags(&d.done, ea::kDeviceEventFlags));
  if ((rc = after_last_use(w, stream)) != EA_OK) return rc;
  // token offsets are the caller's sequence starts, all at most seq_offsets[n]
  const bool wide = seq_offsets[n_seqs] > INT32_MAX || total > INT32_MAX || force_wide();
  const int64_t meta_bytes = offsets_bytes(n_seqs, wide);
  if (meta_bytes > d.cap_meta) {
    // the slot's buffers are free (its event has fired); grow them
    if (d.h_meta) (void)hipHostFree(d.h_meta);
    if (d.d_meta) (void)hipFree(d.d_meta);
    d.h_meta = d.d_meta = nullptr;
    d.cap_meta = 0;
    const int64_t c = std::max<int64_t>(meta_bytes, 1 << 16);
    HS_HIP(hipHostMalloc((void **)&d.h_meta, (size_t)c, hipHostMallocDefault));
    HS_HIP(hipMalloc((void **)&d.d_meta, (size_t)c));
    d.cap_meta = c;
  }
  if (total > d.cap_mid) {
    if (d.d_mid) (void)hipFree(d.d_mid);
    d.d_mid = nullptr;
    d.cap_mid = 0;
    const int64_t c = std::max<int64_t>(total, 4096);
    HS_HIP(hipMalloc((void **)&d.d_mid, (size_t)c * 32));
    d.cap_mid = c;
  }
  put_offsets(d.h_meta, key_offsets_out, seq_offsets, 0, n_seqs, wide);
  HS_HIP(hipMemcpyAsync(d.d_meta, d.h_meta, (size_t)meta_bytes, hipMemcpyHostToDevice, stream));
  const uint8_t *d_koff = d.d_meta;
  const uint8_t *d_toff = d_koff + (n_seqs + 1) * (wide ? 8 : 4);
  if ((rc = run_kernels(d_tokens, d_koff, d_toff, wide, n_seqs, total, block_tokens, d.d_mid,
                        d_parents, d_keys_out, stream)) != EA_OK)
    return rc;
  // one event ends both the slot's use and the workspace's
  HS_HIP(hipEventRecord(d.done, stream));
  d.used = true;
  w.last = d.done;
  w.used = true;
  return EA_OK;
}

namespace {

// Host-side checks of the device-offsets entry points; *key_bound gets the
// most keys the call can produce (the kernels' grid bound).
int check_device_offsets(const int32_t *d_tokens, int64_t n_tokens,
                         const int64_t *d_seq_offsets, int32_t n_seqs, int32_t block_tokens,
                         const uint8_t *d_keys_out, int64_t keys_capacity,
                         const int64_t *d_key_offsets_out, int64_t *key_bound) {
  if (n_tokens < 0 || keys_capacity < 0 || n_seqs < 0) return EA_EINVAL;
  if (!d_seq_offsets || !d_key_offsets_out) return EA_EINVAL;
  const int rc = check_block(block_tokens);
  if (rc != EA_OK) return rc;
  // sequences are consecutive ranges of the n_tokens tokens, so they hold
  // at most n_tokens / b full blocks together
  *key_bound = std::min(keys_capacity, n_tokens / block_tokens);
  if (*key_bound > 0 && (!d_tokens || !d_keys_out)) return EA_EINVAL;
  if (d_keys_out && ((uintptr_t)d_keys_out & 15) != 0) return EA_EINVAL;
  if (((uintptr_t)d_seq_offsets & 7) != 0 || ((uintptr_t)d_key_offsets_out & 7) != 0)
    return EA_EINVAL;
  return EA_OK;
}

}  // namespace

extern "C" int ea_hash_blocks_device_offsets(const int32_t *d_tokens, int64_t n_tokens,
                                             const int64_t *d_seq_offsets, int32_t n_seqs,
                                             int32_t block_tokens, const uint8_t *d_parents,
                                             uint8_t *d_keys_out, int64_t keys_capacity,
                                             int64_t *d_key_offsets_out, hipStream_t stream) {
  int64_t bound = 0;
  int rc = check_device_offsets(d_tokens, n_tokens, d_seq_offsets, n_seqs, block_tokens,
                                d_keys_out, keys_capacity, d_key_offsets_out, &bound);
  if (rc != EA_OK) return rc;
  HashWs *wp = nullptr;
  if ((rc = workspace(stream, &wp)) != EA_OK) return rc;
  HashWs &w = *wp;
  std::lock_guard<std::mutex> lk(w.mu);
  if ((rc = after_last_use(w, stream)) != EA_OK) return rc;
  const bool wide = n_tokens > INT32_MAX || bound > INT32_MAX || force_wide();
  const int64_t off_bytes = offsets_bytes(n_seqs, wide);
  if ((rc = grow_device(w, &w.d_off, &w.cap_off, off_bytes)) != EA_OK) return rc;
  const int64_t scan_bytes = ea::hash_scan_state_bytes(n_seqs);
  if (scan_bytes > w.cap_scan) {
    if ((rc = grow_device(w, &w.d_scan, &w.cap_scan, scan_bytes)) != EA_OK) return rc;
    HS_HIP(ea::launch_hash_scan_reset(w.d_scan, stream));  // a fresh ticket counter
  }
  if ((rc = ensure_mid(w, &w.d_mid, &w.cap_mid, std::max<int64_t>(bound, 1))) != EA_OK) return rc;
  if (bound > 0 && ea::hash_fused(n_seqs)) {  // offsets and keys in two kernels
    HS_HIP(ea::launch_hash_fused_offsets(d_tokens, d_seq_offsets, n_seqs, n_tokens, block_tokens,
                                         bound, d_key_offsets_out, d_parents, d_keys_out,
                                         w.d_scan, stream));
    return release(w, stream, false);
  }
  uint8_t *d_koff = w.d_off;
  uint8_t *d_toff = d_koff + (n_seqs + 1) * (wide ? 8 : 4);
  HS_HIP(ea::launch_hash_key_offsets(d_seq_offsets, n_seqs, n_tokens, block_tokens, bound,
                                     d_key_offsets_out, wide, d_koff, d_toff, w.d_scan, stream));
  if (bound > 0 && n_seqs > 0 &&
      (rc = run_kernels(d_tokens, d_koff, d_toff, wide, n_seqs, bound, block_tokens, w.d_mid,
                        d_parents, d_keys_out, stream)) != EA_OK)
    return rc;
  return release(w, stream, false);
}

extern "C" int ea_hash_blocks_device_offsets_noalloc(
    const int32_t *d_tokens, int64_t n_tokens, const int64_t *d_seq_offsets, int32_t n_seqs,
    int32_t block_tokens, const uint8_t *d_parents, uint8_t *d_keys_out, int64_t keys_capacity,
    int64_t *d_key_offsets_out, hipStream_t stream) {
  int64_t bound = 0;
  int rc = check_device_offsets(d_tokens, n_tokens, d_seq_offsets, n_seqs, block_tokens,
                                d_keys_out, keys_capacity, d_key_offsets_out, &bound);
  if (rc != EA_OK) return rc;
  // the fixed scratch holds this many keys and sequences
  if (bound > ea::kScratchKeys || (int64_t)n_seqs > ea::kScratchSeqs) return EA_EINVAL;
  void *scratch = nullptr;
  HS_HIP(ea::hash_scratch(stream, &scratch));
  uint8_t *base = static_cast<uint8_t *>(scratch);
  const bool wide = n_tokens > INT32_MAX || bound > INT32_MAX || force_wide();
  if (bound > 0 && ea::hash_fused(n_seqs)) {  // offsets and keys in two kernels
    HS_HIP(ea::launch_hash_fused_offsets(d_tokens, d_seq_offsets, n_seqs, n_tokens, block_tokens,
                                         bound, d_key_offsets_out, d_parents, d_keys_out,
                                         base + ea::kScratchState, stream));
    return EA_OK;
  }
  uint8_t *d_koff = base + ea::kScratchOffsets;
  uint8_t *d_toff = d_koff + (n_seqs + 1) * (wide ? 8 : 4);
  HS_HIP(ea::launch_hash_key_offsets(d_seq_offsets, n_seqs, n_tokens, block_tokens, bound,
                                     d_key_offsets_out, wide, d_koff, d_toff,
                                     base + ea::kScratchState, stream));
  if (bound > 0 && n_seqs > 0)
    return run_kernels(d_tokens, d_koff, d_toff, wide, n_seqs, bound, block_tokens,
                       reinterpret_cast<uint32_t *>(base), d_parents, d_keys_out, stream);
  return EA_OK;
}
