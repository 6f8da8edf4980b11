// Hash entry points of libea: chained prefix-block keys on the GPU.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <climits>
#include <cstdint>
#include <cstdlib>
#include <cstring>
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

// Offsets and midstates of one asynchronous (device) call.  Two of them
// alternate, so the host prepares the next call while the GPU runs one.
struct DevSlot {
  uint8_t *h_meta = nullptr, *d_meta = nullptr;
  int64_t cap_meta = 0;
  uint32_t *d_mid = nullptr;
  int64_t cap_mid = 0;  // keys
  hipEvent_t done = nullptr;
  bool used = false;
};

// Grow-only device/pinned buffers for hashing on the current device.
struct HashWs {
  int device = -1;
  hipEvent_t done = nullptr;  // end of the last call's use of the buffers
  bool used = false;
  // pinned host
  uint8_t *h_tok = nullptr;  int64_t cap_tok = 0;   // bytes
  uint8_t *h_meta = nullptr; int64_t cap_meta = 0;  // offsets + parents
  uint8_t *h_keys = nullptr; int64_t cap_keys = 0;  // bytes
  // device
  uint8_t *d_tok = nullptr;
  uint8_t *d_meta = nullptr;
  uint8_t *d_keys = nullptr;
  uint32_t *d_mid = nullptr; int64_t cap_mid = 0;   // keys
  DevSlot slots[2];                                 // ea_hash_blocks_device
  int next = 0;
};

HashWs g_ws;
std::mutex g_ws_mu;

int grow_pair(uint8_t **h, uint8_t **d, int64_t *cap, int64_t need) {
  if (need <= *cap) return EA_OK;
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

int prepare(HashWs &w) {
  int dev;
  HS_HIP(hipGetDevice(&dev));
  if (w.used) HS_HIP(hipEventSynchronize(w.done));
  if (w.device != dev) {
    // buffers belong to one device; drop them when the caller switches
    if (w.h_tok) (void)hipHostFree(w.h_tok);
    if (w.h_meta) (void)hipHostFree(w.h_meta);
    if (w.h_keys) (void)hipHostFree(w.h_keys);
    if (w.d_tok) (void)hipFree(w.d_tok);
    if (w.d_meta) (void)hipFree(w.d_meta);
    if (w.d_keys) (void)hipFree(w.d_keys);
    if (w.d_mid) (void)hipFree(w.d_mid);
    if (w.done) (void)hipEventDestroy(w.done);
    for (DevSlot &d : w.slots) {
      if (d.used) (void)hipEventSynchronize(d.done);
      if (d.h_meta) (void)hipHostFree(d.h_meta);
      if (d.d_meta) (void)hipFree(d.d_meta);
      if (d.d_mid) (void)hipFree(d.d_mid);
      if (d.done) (void)hipEventDestroy(d.done);
    }
    w = HashWs();
    w.device = dev;
  }
  if (!w.done) HS_HIP(hipEventCreateWithFlags(&w.done, hipEventDisableTiming));
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

// Checks the arguments and fills key_offsets_out (running sums of full
// blocks) in one pass over the sequences.
int validate(const int64_t *seq_offsets, int32_t n_seqs, int32_t block_tokens,
             int64_t *key_offsets_out, int64_t *total_keys) {
  if (n_seqs < 0 || !key_offsets_out) return EA_EINVAL;
  if (n_seqs > 0 && !seq_offsets) return EA_EINVAL;
  if (block_tokens < 1 || block_tokens > (1 << 20)) return EA_EINVAL;
  if (block_tokens % 16 != 0) return EA_ENOTSUP;
  const BlockCount blocks(block_tokens);
  int64_t k = 0;
  key_offsets_out[0] = 0;
  for (int32_t s = 0; s < n_seqs; ++s) {
    const int64_t a = seq_offsets[s], e = seq_offsets[s + 1];
    if (a < 0 || e < a) return EA_EINVAL;
    k += blocks(e - a);
    key_offsets_out[s + 1] = k;
  }
  *total_keys = k;
  return EA_OK;
}

int ensure_mid(uint32_t **mid, int64_t *cap, int64_t keys) {
  if (keys <= *cap) return EA_OK;
  if (*mid) (void)hipFree(*mid);
  *mid = nullptr;
  *cap = 0;
  const int64_t c = std::max<int64_t>(keys, 4096);
  HS_HIP(hipMalloc((void **)mid, (size_t)c * 32));
  *cap = c;
  return EA_OK;
}

// Key offsets [n+1] then token offsets [n] for the kernels, written at h as
// int32 when `wide` is false (every value below 2^31: half the bytes to
// upload) and int64 otherwise.  Token offsets are toff[s], or koff[s] * b
// for tokens packed block after block (toff null).  Returns the bytes
// written, rounded up to 16.
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

int64_t offsets_bytes(int32_t n, bool wide) {
  return ((2 * (int64_t)n + 1) * (wide ? 8 : 4) + 15) / 16 * 16;
}

int64_t put_offsets(uint8_t *h, const int64_t *koff, const int64_t *toff, int64_t b, int32_t n,
                    bool wide) {
  if (wide)
    write_offsets<int64_t>(h, koff, toff, b, n);
  else
    write_offsets<int32_t>(h, koff, toff, b, n);
  return offsets_bytes(n, wide);
}

}  // namespace

extern "C" int ea_hash_blocks(const int32_t *tokens, const int64_t *seq_offsets,
                              int32_t n_seqs, int32_t block_tokens,
                              const uint8_t *parents, uint8_t *keys_out,
                              int64_t *key_offsets_out, hipStream_t stream) {
  int64_t total = 0;
  int rc = validate(seq_offsets, n_seqs, block_tokens, key_offsets_out, &total);
  if (rc != EA_OK) return rc;
  if (total > 0 && (!tokens || !keys_out)) return EA_EINVAL;
  if (total == 0) return EA_OK;

  std::lock_guard<std::mutex> lk(g_ws_mu);
  HashWs &w = g_ws;
  if ((rc = prepare(w)) != EA_OK) return rc;
  // pack the full-block tokens of every sequence contiguously
  const int64_t tok_bytes = total * block_tokens * 4;
  const bool wide = total * block_tokens > INT32_MAX || force_wide();
  const int64_t off_bytes = offsets_bytes(n_seqs, wide);
  const int64_t meta_bytes = off_bytes + (parents ? 32 * (int64_t)n_seqs : 0);
  if ((rc = grow_pair(&w.h_tok, &w.d_tok, &w.cap_tok, tok_bytes)) != EA_OK) return rc;
  if ((rc = grow_pair(&w.h_meta, &w.d_meta, &w.cap_meta, meta_bytes)) != EA_OK) return rc;
  if ((rc = grow_pair(&w.h_keys, &w.d_keys, &w.cap_keys, total * 32)) != EA_OK) return rc;
  if ((rc = ensure_mid(&w.d_mid, &w.cap_mid, total)) != EA_OK) return rc;

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
  HS_HIP(ea::launch_sha256_midstates(reinterpret_cast<const int32_t *>(w.d_tok), d_koff,
                                     d_toff, wide, n_seqs, total, block_tokens, w.d_mid,
                                     stream));
  HS_HIP(ea::launch_sha256_chain(w.d_mid, d_koff, wide, n_seqs, block_tokens, d_par, w.d_keys,
                                 stream));
  HS_HIP(hipMemcpyAsync(w.h_keys, w.d_keys, (size_t)total * 32, hipMemcpyDeviceToHost, stream));
  HS_HIP(hipEventRecord(w.done, stream));
  w.used = true;
  HS_HIP(hipEventSynchronize(w.done));
  std::memcpy(keys_out, w.h_keys, (size_t)total * 32);
  return EA_OK;
}

extern "C" int ea_hash_blocks_device(const int32_t *d_tokens, const int64_t *seq_offsets,
                                     int32_t n_seqs, int32_t block_tokens,
                                     const uint8_t *d_parents, uint8_t *d_keys_out,
                                     int64_t *key_offsets_out, hipStream_t stream) {
  int64_t total = 0;
  int rc = validate(seq_offsets, n_seqs, block_tokens, key_offsets_out, &total);
  if (rc != EA_OK) return rc;
  if (total > 0 && (!d_tokens || !d_keys_out)) return EA_EINVAL;
  if (d_keys_out && ((uintptr_t)d_keys_out & 15) != 0) return EA_EINVAL;
  if (total == 0) return EA_OK;

  std::lock_guard<std::mutex> lk(g_ws_mu);
  HashWs &w = g_ws;
  int dev;
  HS_HIP(hipGetDevice(&dev));
  if (w.device != dev && (rc = prepare(w)) != EA_OK) return rc;
  DevSlot &d = w.slots[w.next];
  w.next ^= 1;
  if (d.used) HS_HIP(hipEventSynchronize(d.done));  // the call two back is done
  if (!d.done) HS_HIP(hipEventCreateWithFlags(&d.done, hipEventDisableTiming));
  // token offsets are the caller's sequence starts, all at most seq_offsets[n]
  const bool wide = seq_offsets[n_seqs] > INT32_MAX || total > INT32_MAX || force_wide();
  const int64_t meta_bytes = offsets_bytes(n_seqs, wide);
  if ((rc = grow_pair(&d.h_meta, &d.d_meta, &d.cap_meta, meta_bytes)) != EA_OK) return rc;
  if ((rc = ensure_mid(&d.d_mid, &d.cap_mid, total)) != EA_OK) return rc;
  put_offsets(d.h_meta, key_offsets_out, seq_offsets, 0, n_seqs, wide);
  HS_HIP(hipMemcpyAsync(d.d_meta, d.h_meta, (size_t)meta_bytes, hipMemcpyHostToDevice, stream));
  const uint8_t *d_koff = d.d_meta;
  const uint8_t *d_toff = d_koff + (n_seqs + 1) * (wide ? 8 : 4);
  HS_HIP(ea::launch_sha256_midstates(d_tokens, d_koff, d_toff, wide, n_seqs, total,
                                     block_tokens, d.d_mid, stream));
  HS_HIP(ea::launch_sha256_chain(d.d_mid, d_koff, wide, n_seqs, block_tokens, d_parents,
                                 d_keys_out, stream));
  HS_HIP(hipEventRecord(d.done, stream));
  d.used = true;
  return EA_OK;
}
