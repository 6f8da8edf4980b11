// Internal declarations shared by the host side of libea and its kernels.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace ea {

// Direction of a piece copy: cache pages -> slot-layout buffer (store,
// gather) or slot-layout buffer -> cache pages (load, scatter).
enum CopyDir : int { kToSlots = 0, kToPages = 1 };

// Up to this many entries travel inside the kernel arguments instead of a
// device index array (the small-batch latency path).
constexpr int kInlineMax = 32;

// Flags of events that only order later device work, or tell the host that
// the GPU has finished reading a host buffer: nothing the host reads
// depends on them, so they skip the system-scope release on completion
// (1.4 us added per record between 86 us kernels, against 3.2 us with it).
constexpr unsigned kDeviceEventFlags = hipEventDisableTiming | hipEventDisableSystemFence;

// A slot holds a chunk of `chunk` (C) pages laid out [L][C][piece], then the
// [L][C][8]-byte scale trailer.  Entry i is one page: it goes to chunk
// position i % C of its slot.
struct PieceCopy {
  uint8_t *cache;            // [L][P][piece] bytes
  uint8_t *scales;           // [L][P][8] bytes or nullptr
  uint8_t *slots;            // slot-layout buffer (host mapping or HBM staging)
  const int32_t *pages;      // device [n] or nullptr when inline
  const int64_t *slot_idx;   // device [n] (slot of each entry) or nullptr when
                             // inline / identity
  int64_t n;                 // entries (pages)
  int64_t num_pages;         // P
  int64_t piece_bytes;       // multiple of 16
  int64_t slot_bytes;
  int64_t payload_bytes;     // C * L * piece: offset of the scale trailer
  int32_t num_layers;        // L
  int32_t chunk;             // C >= 1
  int32_t layer_begin;
  int32_t layer_count;
  int32_t identity_slots;    // slot of entry i is i / C (staging buffers)
  int32_t layer_major;       // units ordered layer by layer, else entry by entry
  // Loads first on the host link.  link_flag is the tier's count of load
  // waves at work (nullptr: no priority).  A load (link_role 2) raises it
  // by one per wave for the wave's whole loop; a store (link_role 1) that
  // finds it non-zero sleeps yield_units x 1,024 cycles per 32 KiB it has
  // copied since its last sleep.
  uint32_t *link_flag;
  int32_t link_role;
  int32_t yield_units;
  // Only workgroups on XCDs in xcd_mask do work.  Workgroups of a dispatch
  // go round-robin over the XCDs starting at an offset the hardware chooses
  // (workgroup b runs on XCD (b + offset) % num_xcd), so the workgroup's
  // rank on its XCD is b / num_xcd.  hw_xcd = 1: the XCD is read from the
  // hardware (HW_REG_XCC_ID); 0: it is taken as b % num_xcd, which places
  // the work by luck of the offset but covers every unit all the same.
  int32_t num_xcd;
  uint32_t xcd_mask;
  int32_t hw_xcd;
};

// HBM gather/scatter calls of up to kArgPagesMax pages carry their page ids
// in the kernel arguments (8 KiB) instead of a mapped index buffer: with
// nothing to release after the kernel, back-to-back calls launch with no
// event between them.
constexpr int kArgPagesMax = 2048;
struct ArgPages {
  int32_t pages[kArgPagesMax];
};

struct InlineIdx {
  int32_t pages[kInlineMax];
  int64_t slots[kInlineMax];
};

// Remember the HIP error behind an EA_EHIP return on this thread.
void set_last_hip(int err);

}  // namespace ea
struct ea_tier;
namespace ea {

// A wall-clock controller attaches (on) to or detaches (off) from the tier;
// while at least one is attached the tier reads the steady clock itself for
// decisions, reports and eviction stamps.
void tier_use_steady_clock(ea_tier *t, bool on);
// Count a controller attached to (+1) or detached from (-1) the tier; a tier
// with controllers attached refuses ea_tier_destroy.
void tier_attach_controller(ea_tier *t, int delta);

// Which memory the slot-layout buffer of a piece copy lives in.
enum Route : int { kRouteHostLink = 0, kRouteHbm = 1 };
// PieceCopy::link_role
enum LinkRole : int { kLinkNone = 0, kLinkYield = 1, kLinkMark = 2 };

// Check, with a probe kernel on the current device, that the workgroups of
// a dispatch go round-robin over num_xcd XCDs as the hardware reports them
// (the property the hardware-placed piece copies rely on).  *ok = false
// when any probe dispatch breaks it.
hipError_t probe_xcd_round_robin(int num_xcd, bool *ok);

// Launch one piece-copy kernel with at most `workgroups` (> 0) working
// workgroups, placed on the XCDs of a.xcd_mask.
// The entries' indices come from inl (at most kInlineMax, in the arguments),
// ids (page ids of at most kArgPagesMax entries of an HBM copy with
// identity slots, in the arguments) or, with both null, a.pages and
// a.slot_idx.
hipError_t launch_piece_copy(const PieceCopy &a, const InlineIdx *inl, const ArgPages *ids,
                             int dir, int route, int64_t workgroups, hipStream_t stream);

// Add delta to a tier's load counter on `stream` (a one-lane kernel).

// XOR checksum of one layer's piece of each of n pages (device page ids).
hipError_t launch_layer_checksum(const uint8_t *cache, const uint8_t *scales, int64_t num_pages,
                                 int64_t piece_bytes, int32_t layer, const int32_t *pages,
                                 int32_t n, uint64_t *out, hipStream_t stream);

// SHA-256 chained keys.
//  mid:  device [n_keys][8] words scratch
//  d_key_offsets: device [n_seqs+1] key offsets; d_tok_offsets: device
//  [n_seqs] token offset of each sequence; both int32 when `wide` is false
//  (every offset below 2^31), int64 when it is true.
hipError_t launch_sha256_midstates(const int32_t *d_tokens, const void *d_key_offsets,
                                   const void *d_tok_offsets, bool wide, int32_t n_seqs,
                                   int64_t n_keys, int32_t block_tokens, uint32_t *d_mid,
                                   hipStream_t stream);
hipError_t launch_sha256_chain(const uint32_t *d_mid, const void *d_key_offsets, bool wide,
                               int32_t n_seqs, int32_t block_tokens, const uint8_t *d_parents,
                               uint8_t *d_keys, hipStream_t stream);

// The one-kernel form for large batches (a lane per sequence computes its
// keys' token blocks and chained blocks in turn): chosen when there are at
// least 256 sequences per compute unit, or forced with EA_HASH_CHAIN=fused
// (any other EA_HASH_CHAIN value keeps the two kernels).
bool hash_fused(int32_t n_seqs);
hipError_t launch_sha256_fused(const int32_t *d_tokens, const void *d_key_offsets,
                               const void *d_tok_offsets, bool wide, int32_t n_seqs,
                               int32_t block_tokens, const uint8_t *d_parents, uint8_t *d_keys,
                               hipStream_t stream);

// Key offsets from device sequence offsets d_seq_offsets [n_seqs+1], in two
// kernels: d_key_offsets_out [n_seqs+1] (int64) and the hash kernels'
// copies d_koff [n_seqs+1], d_toff [n_seqs] (int32 unless wide).  On
// invalid offsets, or more than keys_cap keys, d_key_offsets_out[0] = -1
// and d_koff is all zero (the hash kernels then write nothing).  d_state:
// hash_scan_state_bytes(n_seqs) bytes of device memory whose first 8 bytes
// are zero before the call (the kernels leave them zero again).
hipError_t launch_hash_key_offsets(const int64_t *d_seq_offsets, int32_t n_seqs,
                                   int64_t n_tokens, int32_t block_tokens, int64_t keys_cap,
                                   int64_t *d_key_offsets_out, bool wide, void *d_koff,
                                   void *d_toff, void *d_state, hipStream_t stream);
// The same offsets and the keys for batches that take the fused form
// (hash_fused): the scan's first kernel, then one kernel that scans each
// workgroup's sequences from its prefix, writes d_key_offsets_out and
// hashes.  Same failure contract; d_state as above.
hipError_t launch_hash_fused_offsets(const int32_t *d_tokens, const int64_t *d_seq_offsets,
                                     int32_t n_seqs, int64_t n_tokens, int32_t block_tokens,
                                     int64_t keys_cap, int64_t *d_key_offsets_out,
                                     const uint8_t *d_parents, uint8_t *d_keys, void *d_state,
                                     hipStream_t stream);
int64_t hash_scan_groups(int32_t n_seqs);
// Zero the first 8 bytes of a scan state on `stream` (a fill kernel).
hipError_t launch_hash_scan_reset(void *d_state, hipStream_t stream);

// The fixed device memory of the hashing entry point that allocates
// nothing, per device: midstates of up to kScratchKeys keys, the kernels'
// key and token offsets (64-bit) of up to kScratchSeqs sequences, then the
// scan state.  48 MiB in all.
constexpr int64_t kScratchKeys = int64_t(1) << 20;
constexpr int64_t kScratchSeqs = int64_t(1) << 20;
constexpr int64_t kScratchOffsets = 32 * kScratchKeys;  // byte offsets in the scratch
constexpr int64_t kScratchState = kScratchOffsets + (8 * (2 * kScratchSeqs + 1) + 255) / 256 * 256;
// Sequences per workgroup of the key-offset scan, and per sub-block of it
// (the fused hash kernel's workgroups, one sequence per work-item).  The
// scan state holds 64 bytes, two words per group and one per sub-block.
constexpr int64_t kHashScanSeqs = 2048;
constexpr int64_t kHashScanSub = 256;
constexpr int64_t hash_scan_state_for(int64_t groups) {
  return 64 + 16 * groups + 8 * groups * (kHashScanSeqs / kHashScanSub);
}
constexpr int64_t kScratchBytes =
    kScratchState + hash_scan_state_for((kScratchSeqs + kHashScanSeqs - 1) / kHashScanSeqs);
// The scratch's address on the current device: resolved with
// hipGetSymbolAddress the first time a device asks (that device current),
// then kept; the first resolution also zeroes the scan's ticket counter
// with a fill kernel on `stream`.
hipError_t hash_scratch(hipStream_t stream, void **ptr);
inline int64_t hash_scan_state_bytes(int32_t n_seqs) {
  return hash_scan_state_for(hash_scan_groups(n_seqs));
}


}  // namespace ea
