/*
 * ea.h -- C ABI of the MI355X KV-offload library (libea.so).
 *
 * The library moves KV cache state between a paged GPU cache in HBM and a
 * pinned host-memory tier, as described in "EfficientAgent: What Makes KV
 * Cache Offloading Work for Concurrent Agents?" (arXiv 2609.33762): host
 * writes and restores are KV copied from GPU to host and back (section 2, "A
 * closed-loop workload"); reusable prefixes are found through chained
 * content keys of full blocks (section 2 "Exact-prefix reuse", section 3.2);
 * and a write-admission rule decides, once per request, whether its new KV
 * enters the tier (section 4, Eq. 6; App. "Runtime Admission Details",
 * Eq. 10), with copy-time deduplication.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Return value: EA_OK (0) or a negative EA_E* code.  ea_strerror() gives
 *    text; ea_last_hip_error() gives the HIP error behind EA_EHIP on this
 *    thread.
 *  - Arguments are validated before anything is enqueued: on any error no
 *    byte moves and no tier metadata changes.
 *  - Index arrays (block ids, slots, masks, keys) are HOST pointers and are
 *    read before the call returns; the caller may reuse them at once.
 *  - Copies are asynchronous on the caller's HIP stream and ordered with the
 *    caller's other work on that stream.  A store or load that touches a host
 *    slot that an earlier call on another stream still transfers waits for
 *    that transfer on the device (no host blocking).  A store and a load
 *    share the host link in both directions at once only when their streams
 *    run on different hardware queues: the HIP runtime places each stream on
 *    one of GPU_MAX_HW_QUEUES queues, and two streams on one queue run one
 *    after the other.  Create the copy streams after the process has first
 *    used the default stream, and keep the streams in use within the
 *    hardware queues.
 *  - GPU cache layout (caller-owned device memory): element array
 *    [L][P][2][T][H][D] of elem_bytes each, so the K and V data of one
 *    (layer, page) form one contiguous "piece" of 2*T*H*D*elem_bytes bytes.
 *    The optional scale plane is a caller-owned float32 array [L][P][2]
 *    (K scale, V scale of each layer and page), moved as opaque bytes.
 *  - Host slot layout (library-owned pinned memory): slot s holds one chunk
 *    of C = chunk_pages pages (C = 1 unless the tier was created with
 *    ea_tier_create_chunked) of every layer, [L][C][2][T][H][D], so one layer
 *    of a chunk is contiguous, followed when scales exist by an [L][C][2]
 *    float32 trailer padded to a multiple of 256 bytes.  The tier holds
 *    K_H = floor(capacity_bytes / slot_bytes) slots; each has one key.
 *  - A tier is internally locked; one tier may be used from several threads.
 *    Calls are bound to the device that was current when the cache or tier
 *    was created.
 *
 * Environment variables (tuning and testing; the defaults are the measured
 * best on MI355X, and every setting gives the same bytes and keys)
 * -------------------------------------------------------------------------
 *  EA_TRANSFER=direct|staged   transfer plan of tiers left at EA_PLAN_AUTO
 *  EA_LINK_WG, EA_LINK_WG_STORE, EA_LINK_WG_LOAD
 *                              working workgroups of a direct store / load
 *                              (8 / 8; EA_LINK_WG sets both)
 *  EA_LOAD_PRIORITY            sleep (in units of 1,024 cycles) a direct
 *                              store's waves take per 32 KiB copied while
 *                              waves of a direct or layered load of the same
 *                              tier run (31; 0 = off); read at tier creation
 *  EA_LINK_WG_LAYERED          workgroups of one layer of a layered load (16)
 *  EA_XCD_STORE, EA_XCD_LOAD   XCD masks of the two directions (0x5, 0xA
 *                              with four or more XCDs); read at tier creation
 *  EA_XCD_PLACEMENT=index      place work by workgroup index, not by the XCD
 *                              the hardware reports; read at cache creation
 *  EA_GRID_HBM, EA_GRID_GATHER, EA_GRID_SCATTER
 *                              workgroups of the HBM gather (512) / scatter (256)
 *  EA_HBM_ORDER, EA_GATHER_ORDER, EA_SCATTER_ORDER = entry|layer
 *                              unit order of the HBM gather / scatter: each
 *                              page's layers in turn (entry, the default) or
 *                              one layer of every page at a time
 *  EA_HBM_INDEX=ring           page ids of an HBM gather / scatter (and of
 *                              the staged plan's) through the mapped index
 *                              ring even for 33-2,048 pages, which by default
 *                              travel in the kernel arguments
 *  EA_STAGING_MB               HBM staging of the staged plan per direction (512)
 *  EA_HOST_COHERENT=0          non-coherent pinned memory for new tiers
 *  EA_HOST_ALLOC_WAIT_MS       how long a tier's failed pinned allocation is
 *                              retried (5000; 0 = fail at once)
 *  EA_HASH_CHAIN=split|pair|lane, EA_HASH_MID=split|lane
 *                              force a form of the hash kernels
 *  EA_HASH_OFFSETS=64          64-bit offsets for the hash kernels
 */
#ifndef EA_H
#define EA_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  EA_OK = 0,
  EA_EINVAL = -1,  /* bad argument: null pointer, out-of-range id or slot,
                      duplicate destination, unsupported shape               */
  EA_ENOMEM = -2,  /* host or device allocation failed                      */
  EA_ENOSPC = -3,  /* reserved: no tier call fails for lack of space; a full
                      tier reports unallocated blocks instead                */
  EA_EHIP = -4,    /* a HIP call failed; see ea_last_hip_error()            */
  EA_ENOTSUP = -5  /* valid request the library does not implement        */
};

const char *ea_strerror(int code);
int ea_last_hip_error(void);

/* ------------------------------------------------------------------ cache */

typedef struct {
  void *base;           /* device pointer, [L][P][2][T][H][D], 16-B aligned  */
  void *scale_base;     /* device pointer to [L][P][2] float32, or NULL      */
  int32_t num_pages;    /* P                                                  */
  int32_t num_layers;   /* L                                                  */
  int32_t page_tokens;  /* T, tokens per page (one hash block)               */
  int32_t num_kv_heads; /* H, KV heads held by this rank                     */
  int32_t head_dim;     /* D                                                  */
  int32_t elem_bytes;   /* bytes per element: 2 for bf16, 1 for fp8          */
} ea_cache_desc;

typedef struct ea_cache ea_cache;

/* Describe a caller-owned paged KV cache (KV footprint of Eq. 1: a page of
 * T tokens holds T * 2 * L * D * elem_bytes * H bytes).  The piece size
 * 2*T*H*D*elem_bytes must be a multiple of 16 bytes (EA_EINVAL otherwise).
 * The library never frees base or scale_base. */
int ea_cache_create(const ea_cache_desc *desc, ea_cache **out);
int ea_cache_destroy(ea_cache *cache);

/* ------------------------------------------------------------------- tier */

typedef struct ea_tier ea_tier;

typedef struct {
  int64_t capacity_slots; /* K_H                                              */
  int64_t slot_bytes;
  int64_t piece_bytes;
  int64_t page_bytes;     /* data bytes of a slot (trailer excluded): C*L*piece */
  int64_t trailer_bytes;
  int64_t capacity_bytes; /* C_H as given at creation                         */
  void *host_base;        /* host address of slot 0 (pinned, mapped)          */
  void *device_base;      /* the same memory as seen by kernels               */
  int64_t chunk_pages;    /* C: pages per slot                                */
} ea_tier_info;

/* Create the host tier: K_H = floor(capacity_bytes / slot_bytes) slots of
 * pinned, device-mapped host memory, OWNED by the library (freed by
 * ea_tier_destroy).  `shape` supplies the slot layout (the tier can serve
 * any cache of the same shape).  numa_node >= 0 binds the allocation to that
 * NUMA node; -1 uses the runtime's default placement.  capacity_bytes is also
 * the C_H the write rule compares the working-set estimate with.  Fails with
 * EA_EINVAL if K_H < 1, EA_ENOMEM if the pinned allocation fails.  The driver
 * returns the pages of a freed tier to its pool only after a delay, so an
 * out-of-memory failure is retried with growing waits for up to
 * EA_HOST_ALLOC_WAIT_MS (5 s by default) before EA_ENOMEM; a request beyond
 * the machine's physical memory fails at once. */
int ea_tier_create(const ea_cache *shape, int64_t capacity_bytes,
                   int numa_node, ea_tier **out);

/* The same with host chunks of chunk_pages (C >= 1) pages: one key, one LRU
 * entry and one slot per chunk (the paper's host chunk of 1,024 tokens is
 * C = 64 pages of 16 tokens, 24 MiB per rank at TP8: Table "Serving
 * configuration").  Keys then come from ea_hash_blocks with block_tokens =
 * C * page_tokens, and stores and loads take C page ids per slot. */
int ea_tier_create_chunked(const ea_cache *shape, int32_t chunk_pages,
                           int64_t capacity_bytes, int numa_node,
                           ea_tier **out);

/* Waits for every transfer the library issued on this tier, then frees it.
 * EA_EINVAL (and nothing freed) while an ea_controller is attached to it. */
int ea_tier_destroy(ea_tier *tier);

int ea_tier_get_info(const ea_tier *tier, ea_tier_info *info);

/* --------------------------------------------------------- chained hashing */

/* Chained prefix-block keys (section 2 "Exact-prefix reuse"; section 3.2: a
 * full chunk's key depends on its entire prefix, so equal text after a
 * different prefix gets a different key and an early edit rekeys every later
 * chunk).  For sequence s = tokens[seq_offsets[s] .. seq_offsets[s+1]) and
 * b = block_tokens, with key_{-1} = parents[s] (32 zero bytes if parents is
 * NULL), every FULL block i gets
 *     key_i = SHA-256( LE32(tok[i*b]) || ... || LE32(tok[i*b+b-1]) || key_{i-1} )
 * (FIPS 180-4 SHA-256; a token is its 32-bit two's-complement value).  A
 * trailing partial block gets no key.
 *
 * Host pointers: tokens int32[seq_offsets[n_seqs]] (only the ranges named by
 * seq_offsets are read), seq_offsets int64[n_seqs+1] non-decreasing from
 * >= 0, parents uint8[n_seqs][32] or NULL; outputs keys_out
 * uint8[sum floor(len_s/b)][32] and key_offsets_out int64[n_seqs+1]
 * (key_offsets_out[0] = 0).  Runs on `stream` and returns when the keys are
 * in keys_out (the scheduler needs them at once, App. "Runtime Admission
 * Details").  block_tokens must be a positive multiple of 16 (EA_ENOTSUP
 * otherwise: the GPU splits each key into 4*b/64 parallel message blocks and
 * one chained block). */
int ea_hash_blocks(const int32_t *tokens, const int64_t *seq_offsets,
                   int32_t n_seqs, int32_t block_tokens,
                   const uint8_t *parents, uint8_t *keys_out,
                   int64_t *key_offsets_out, hipStream_t stream);

/* The same keys from DEVICE-resident tokens: d_tokens (device int32, n_tokens
 * of them), seq_offsets (HOST int64[n_seqs+1]; seq_offsets[n_seqs] <=
 * n_tokens), d_parents (device uint8[n_seqs][32] or NULL), d_keys_out
 * (device uint8[keys_capacity][32], 16-byte aligned) and key_offsets_out
 * (HOST int64[n_seqs+1], filled before return).  EA_EINVAL, nothing
 * launched, when the offsets run past n_tokens or the keys would not fit in
 * keys_capacity.  Asynchronous: the keys are valid once the work enqueued on
 * `stream` completes.
 *
 * Both entry points run the chained compression in one of three forms (the
 * keys are the same): a workgroup of two waves per four sequences while
 * there are at most eight sequences per compute unit, two lanes per sequence
 * up to 32 sequences per SIMD, one lane per sequence beyond; EA_HASH_CHAIN=split,
 * pair or lane forces a form.  The token blocks of keys of 32 tokens or more
 * run in a workgroup of two waves per four keys while there are at most 16
 * keys per compute unit (8 with 32-token keys), one lane per key beyond;
 * EA_HASH_MID=split or lane forces a form.
 * Sequence and key offsets travel to the kernels as 32-bit values when all
 * fit, else as 64-bit values; EA_HASH_OFFSETS=64 forces the latter.
 * Buffers are kept per (device, stream): calls on different streams run
 * concurrently, from any threads. */
int ea_hash_blocks_device(const int32_t *d_tokens, int64_t n_tokens,
                          const int64_t *seq_offsets, int32_t n_seqs,
                          int32_t block_tokens, const uint8_t *d_parents,
                          uint8_t *d_keys_out, int64_t keys_capacity,
                          int64_t *key_offsets_out, hipStream_t stream);

/* The same with the sequence offsets on the DEVICE too, so that nothing
 * crosses the host link: d_seq_offsets (device int64[n_seqs+1], 8-byte
 * aligned) and d_key_offsets_out (device int64[n_seqs+1]).  A kernel derives
 * the key offsets on the device (key_offsets[s] = sum over earlier
 * sequences of floor(len/b)).  The host cannot see the offsets, so
 * malformed ones (a negative start, a decrease, an end past n_tokens) or
 * more keys than keys_capacity are reported on the device: the call then
 * sets d_key_offsets_out[0] = -1 and writes no key.  On success
 * d_key_offsets_out[0] = 0 and d_key_offsets_out[n_seqs] is the key count.
 * Keys need the first lookup of a request at once (App. "Runtime Admission
 * Details"); this form suits callers whose prompts already sit in HBM. */
int ea_hash_blocks_device_offsets(const int32_t *d_tokens, int64_t n_tokens,
                                  const int64_t *d_seq_offsets, int32_t n_seqs,
                                  int32_t block_tokens, const uint8_t *d_parents,
                                  uint8_t *d_keys_out, int64_t keys_capacity,
                                  int64_t *d_key_offsets_out, hipStream_t stream);

/* For callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): ea_hash_blocks_device_
 * offsets with every buffer of its own in fixed device memory that the
 * library reserves per device (48 MiB, held until the process ends), so the
 * call allocates nothing.  Same arguments and results.  Limits: at most
 * 1,048,576 keys (min(keys_capacity, n_tokens / block_tokens)) and
 * 1,048,576 sequences per call, else EA_EINVAL with nothing launched.  All
 * calls on one device share that memory and each leaves it as it found it:
 * two calls that overlap on one device (on different streams, not ordered
 * by events) race and may compute wrong keys; order them. */
int ea_hash_blocks_device_offsets_noalloc(const int32_t *d_tokens, int64_t n_tokens,
                                          const int64_t *d_seq_offsets, int32_t n_seqs,
                                          int32_t block_tokens, const uint8_t *d_parents,
                                          uint8_t *d_keys_out, int64_t keys_capacity,
                                          int64_t *d_key_offsets_out, hipStream_t stream);

/* ------------------------------------------------- lookup and admission */

/* Consecutive-prefix lookup (section 3.2; App. "Prefix coverage from a
 * reference stream"): *hit_blocks = largest k such that keys 0..k-1 are all
 * resident; a lookup stops at the first absent key (a key whose store has
 * not been issued yet counts as absent).  The hits move to the most-recent
 * end of the LRU order in increasing position order (App. "Recency order of
 * the host tier") and each gets one pin, so it cannot be evicted before the
 * caller's load is issued; release with ea_tier_unpin.  slots_out[i] gets the
 * slot of key i for i < *hit_blocks.  keys: host uint8[n][32]. */
int ea_tier_lookup(ea_tier *tier, const uint8_t *keys, int64_t n,
                   int64_t *hit_blocks, int64_t *slots_out);

enum { EA_ADMIT_CONDITIONED = 0, /* Eq. 6 with the pressure signal p_t       */
       EA_ADMIT_ALWAYS = 1,      /* p_t = 0: offload without write admission */
       EA_ADMIT_FIXED = 2 };     /* p_t = 1: fixed write admission           */

typedef struct {
  int64_t theta_ppm;       /* occupancy threshold theta in parts per million
                              (950000 = 0.95): full when
                              registered * 10^6 >= theta_ppm * K_H            */
  int64_t kappa;           /* write threshold in full blocks (u > kappa)      */
  int64_t block_tokens;    /* b                                               */
  int64_t beta_rank;       /* KV bytes per token per rank (Eq. 1)             */
  int64_t activity_window; /* window of A_t and e_t in caller clock units; an
                              event at time t counts when t > now - window    */
  int32_t length_window;   /* N_t = mean n of the last this-many first lookups*/
                           /* Memory stays bounded: once the tier holds more
                              than 65,536 lookups (or eviction stamps) it
                              keeps only those that the largest activity,
                              report and length windows given so far can
                              still reach; a window larger than all earlier
                              ones then sees no events older than they did.   */
  int32_t mode;            /* EA_ADMIT_*                                      */
  int32_t telemetry;       /* 1: the tier's own state is a fresh report;
                              0: no report, the estimate alone decides        */
  int32_t _pad;
} ea_policy;

typedef struct {
  int64_t n_tokens; /* n, prompt tokens                                       */
  int64_t h_tokens; /* h, prompt tokens the host tier already holds           */
  int64_t task_id;  /* agent / task identity (for A_t)                        */
  int64_t now;      /* caller clock; not below the previous first lookup's    */
  int32_t decided;  /* -1: first lookup, decide now and enter the windows;
                       0 or 1: a later lookup of the same request keeps that
                       earlier decision (App. "Runtime Admission Details")    */
  int32_t _pad;
} ea_request;

/* Write admission and copy-time deduplication (section 4, Eq. 6; Eq. 10).
 * With u = floor(n/b) - floor(h/b), A_t = distinct task_ids of the first
 * lookups inside the window (this one included), N_t = mean n of the last
 * length_window first lookups, C_reuse = (A_t - 1) * N_t * beta_rank (Eq. 5)
 * compared exactly with C_H = the tier's capacity_bytes:
 *   p_t  = [C_reuse > C_H] and [registered >= theta K_H and e_t > 0]
 *          (the second factor is dropped when telemetry == 0),
 *   save = not (p_t and u > kappa),
 *   mask_out[i] = save and the tier holds no slot under key i (pending or
 *                 resident: deduplication sees allocations whose store is
 *                 not issued yet).
 * registered counts the chunks whose store has been issued (a store
 * allocates its buffers before it registers the chunks, App. "Runtime
 * Admission Details"), so another request's pending allocation does not
 * raise the occupancy o_t.
 * e_t counts evictions made to allocate inside the window.  n_keys must be
 * floor(n/b); keys host uint8[n_keys][32]; mask_out host uint8[n_keys]. */
int ea_admission_fill(ea_tier *tier, const ea_policy *policy,
                      const ea_request *request, const uint8_t *keys,
                      int64_t n_keys, uint8_t *mask_out, int32_t *save_out);

/* ------------------------------------------------- published telemetry
 *
 * The paper splits the rule between the worker that owns the tier and the
 * scheduler that decides (App. "Runtime Admission Details"): the worker
 * publishes a report every second, the scheduler reads the latest one every
 * half second and uses it only while it is fresh (at most 5 s old); without
 * a fresh report the working-set estimate alone decides. */
typedef struct {
  int64_t time;            /* clock value the report was taken at             */
  int64_t registered;      /* chunks whose store has been issued: the o_t
                              numerator (a store allocates its buffers before
                              it registers its chunks, so pending allocations
                              do not count)                                   */
  int64_t capacity_slots;  /* K_H                                             */
  int64_t evictions;       /* e_t: evictions made to allocate with a stamp in
                              (time - window, time]                           */
} ea_tier_report;

/* Take the tier's report at time `now` (caller clock, not below the tier's
 * clock) over `window`, and advance the tier's clock to `now` (evictions are
 * stamped with the tier's clock: the latest time a decision or a report gave
 * it).  EA_EINVAL if now is earlier than the clock or window < 0. */
int ea_tier_publish(ea_tier *tier, int64_t now, int64_t window,
                    ea_tier_report *out);

/* ea_admission_fill with the "full and evicting" factor taken from the
 * scheduler's copy of a report (Eq. 10): used when policy->telemetry is 1,
 * report is not NULL and 0 <= request->now - report->time <= max_age;
 * otherwise the working-set estimate alone decides.  report may be NULL;
 * max_age >= 0.  Everything else is as in ea_admission_fill. */
int ea_admission_fill_report(ea_tier *tier, const ea_policy *policy,
                             const ea_request *request,
                             const ea_tier_report *report, int64_t max_age,
                             const uint8_t *keys, int64_t n_keys,
                             uint8_t *mask_out, int32_t *save_out);

/* -------------------------------------------------- wall-clock controller
 *
 * The same split as a runtime: a controller attached to a tier publishes
 * its report every report_interval, refreshes the scheduler's copy every
 * read_interval (the copy is the latest report published at or before that
 * read), and decides requests on a microsecond clock with A_t and e_t over
 * `window` (App. "Runtime Admission Details", Table "Write-admission
 * parameters": 1 s, 0.5 s, 5 s, 60 s).  Ticks fall at k * interval after
 * creation (k >= 1); a publish and a read at the same time publish first.
 * With manual_clock = 0 a background thread publishes on the steady clock,
 * decisions take the steady clock, and the tier stamps its evictions with
 * it: decide through the controller only.  With manual_clock = 1 no thread
 * runs and ea_controller_advance moves the clock (creation is time 0), which
 * makes every decision reproducible. */
typedef struct {
  int64_t report_interval; /* microseconds, > 0 (paper: 1,000,000)           */
  int64_t read_interval;   /* microseconds, > 0 (paper: 500,000)             */
  int64_t max_report_age;  /* microseconds, >= 0 (paper: 5,000,000)          */
  int64_t window;          /* microseconds, >= 0, A_t and e_t (paper: 60 s)  */
  int32_t manual_clock;    /* 0: steady clock and a publisher thread          */
  int32_t _pad;
} ea_controller_config;

typedef struct ea_controller ea_controller;

typedef struct {
  int64_t now;                 /* the controller's clock                      */
  int64_t reports_published;
  ea_tier_report published;    /* the last report published                   */
  ea_tier_report seen;         /* the scheduler's copy (valid if have_seen)   */
  int32_t have_seen;
  int32_t fresh;               /* the copy is fresh at `now`                  */
  int64_t decisions;           /* first lookups decided                       */
  int64_t skips;               /* of those, writes declined                   */
  int64_t fresh_decisions;     /* of those, decided with a fresh report       */
} ea_controller_status;

/* policy is copied, with its activity_window replaced by config->window.
 * The tier must outlive the controller: ea_tier_destroy refuses a tier with
 * controllers attached. */
int ea_controller_create(ea_tier *tier, const ea_policy *policy,
                         const ea_controller_config *config,
                         ea_controller **out);
/* Stops and joins the publisher thread, then frees the controller. */
int ea_controller_destroy(ea_controller *ctl);
/* Manual clock only: run every publish and read due up to `now` (not below
 * the controller's clock), then set the clock to `now`. */
int ea_controller_advance(ea_controller *ctl, int64_t now);
/* The write rule at a request's first prefix lookup (decided = -1), or a
 * later lookup of the same request keeping its choice (0 or 1), at the
 * controller's clock, with the scheduler's copy of the report; fills the
 * deduplicated mask like ea_admission_fill_report. */
int ea_controller_decide(ea_controller *ctl, int64_t n_tokens, int64_t h_tokens,
                         int64_t task_id, int32_t decided, const uint8_t *keys,
                         int64_t n_keys, uint8_t *mask_out, int32_t *save_out);
int ea_controller_get_status(ea_controller *ctl, ea_controller_status *out);

/* Allocate host slots for the keys with mask[i] != 0 (mask NULL = all) that
 * the tier does not hold yet (pending or resident): the lowest-numbered free
 * slot, else the least-recent resident slot that no lookup, allocation or transfer pins (an
 * eviction inside allocation, App. "Runtime Admission Details").  New slots
 * are registered under their key, go to the most-recent end in increasing
 * position order, and carry one pin; they become visible to lookups, and
 * count as registered chunks, once ea_store_blocks has been issued for them.  slots_out[i] = -1 where no slot
 * was allocated; once no victim is left every later block gets -1 (not an
 * error).  *allocated gets the number of slots allocated. */
int ea_tier_alloc(ea_tier *tier, const uint8_t *keys, const uint8_t *mask,
                  int64_t n, int64_t *slots_out, int64_t *allocated);

/* Drop one pin from each listed slot (pins from ea_tier_lookup or
 * ea_tier_alloc): the end of a pending lookup or transfer, after which App.
 * "Runtime Admission Details" lets eviction take the chunk again.  A slot
 * allocated but never stored whose last pin goes away is released (the
 * paper does not say what happens to an abandoned allocation).  EA_EINVAL
 * (and no change) if any slot would drop below zero. */
int ea_tier_unpin(ea_tier *tier, const int64_t *slots, int64_t n);

typedef struct {
  int64_t capacity_slots;   /* K_H                                          */
  int64_t allocated;        /* slots holding a key: pending + resident      */
  int64_t registered;       /* resident chunks (store issued): o_t numerator*/
  int64_t pinned;           /* slots with at least one pin                  */
  int64_t evictions_total;  /* evictions made to allocate                   */
  int64_t evictions_window; /* of those, inside the last decision's window  */
  int64_t clock;            /* last first-lookup clock                      */
  int64_t active_tasks;     /* A_t of the last decision                     */
  double mean_prompt;       /* N_t of the last decision (report only)       */
  double working_set;       /* C_reuse of the last decision (report only)   */
  int32_t last_pressure;    /* p_t of the last decision                     */
  int32_t last_save;
  int64_t bytes_stored;     /* bytes enqueued host-ward by ea_store_blocks  */
  int64_t bytes_loaded;     /* bytes enqueued device-ward by loads          */
  int64_t store_calls;
  int64_t load_calls;
} ea_tier_stats_t;

/* Tier telemetry (App. "Runtime Admission Details": registered chunks, K_H,
 * evictions in the window). */
int ea_tier_stats(const ea_tier *tier, ea_tier_stats_t *stats);

enum { EA_SLOT_FREE = 0, EA_SLOT_PENDING = 1, EA_SLOT_RESIDENT = 2 };

/* Full metadata image: per slot its state, pin count and key (zeros when
 * free), and the pending and resident slots from least to most recent in lru_out
 * (*n_lru entries).  Host arrays of K_H entries. */
int ea_tier_export(const ea_tier *tier, uint8_t *state_out, int32_t *pins_out,
                   uint8_t *keys_out, int64_t *lru_out, int64_t *n_lru);

/* ---------------------------------------------------------------- copies */

/* Store ("KV copied from GPU to host", section 2): for every i < n with
 * admit_mask[i] != 0 (NULL = all), host slot host_slots[i] receives pages
 * block_ids[i*C .. i*C+C-1] of every layer (K and V), page i*C+c at chunk
 * position c, and, with scales, their scales as its trailer (then zeros).
 * block_ids has n*C entries (C = the tier's chunk_pages), host_slots and
 * admit_mask n.  Admitted slots must be distinct and in [0, K_H); ids in
 * [0, P) (they may repeat).  Slots allocated by ea_tier_alloc become
 * resident.  The cache must have the tier's shape.  Absent chunks of one
 * request usually get consecutive slots (lowest free first), so a store
 * writes long contiguous runs of host memory (App. "Runtime Admission
 * Details": deduplication passes runs of absent chunks to the store). */
int ea_store_blocks(ea_cache *cache, ea_tier *tier, const int32_t *block_ids,
                    const int64_t *host_slots, const uint8_t *admit_mask,
                    int32_t n, hipStream_t stream);

/* Load (host restore, the T_load of Eq. 2): pages dst_pages[i*C .. i*C+C-1]
 * of every layer receive the chunk in host slot host_slots[i] (chunk
 * position c into page dst_pages[i*C+c], with its scales).  host_slots has
 * n entries, dst_pages n*C.  Destination pages must be distinct; sources may
 * repeat. */
int ea_load_blocks(ea_tier *tier, ea_cache *cache, const int64_t *host_slots,
                   const int32_t *dst_pages, int32_t n, hipStream_t stream);

/* Layer-pipelined load (not in the paper, which restores a prefix as one
 * transfer; it gives the same end state as ea_load_blocks, the restore of
 * Eq. 2, issued one layer at a time so that attention over layer l can
 * start before later layers arrive): on copy_stream, after layer l's copy
 * the library records layer_done[l] (caller-created events; n_events must
 * equal the cache's num_layers, else EA_EINVAL), so a consumer stream can
 * hipStreamWaitEvent(layer_done[l]) and use layer l of every destination
 * page while later layers are still in flight. */
int ea_load_blocks_layered(ea_tier *tier, ea_cache *cache,
                           const int64_t *host_slots, const int32_t *dst_pages,
                           int32_t n, hipStream_t copy_stream,
                           hipEvent_t *layer_done, int32_t n_events);

/* Paged gather / scatter between the cache and a DEVICE buffer in the slot
 * layout of one page per slot.  Not in the paper: they are the HBM half of
 * the staged transfer plan (the GPU-side copy of "KV copied from GPU to
 * host and back", section 2), also usable on their own.
 * gather writes page block_ids[i] (with scales) to d_dst + i*slot_bytes;
 * scatter writes d_src + i*slot_bytes into page dst_pages[i] (destinations
 * distinct).  slot_bytes is that of a tier of the same shape with C = 1;
 * dst_bytes / src_bytes give the device buffer's size, which must hold n
 * slots (EA_EINVAL otherwise, nothing launched).  block_ids / dst_pages are
 * HOST arrays the call has copied by the time it returns (up to 2,048 ids
 * into the kernel arguments, more into the library's mapped index ring), so
 * the caller may reuse them at once; the copy itself is asynchronous on
 * `stream`. */
int ea_gather_blocks(ea_cache *cache, const int32_t *block_ids, int32_t n,
                     void *d_dst, int64_t dst_bytes, hipStream_t stream);
int ea_scatter_blocks(ea_cache *cache, const void *d_src, int64_t src_bytes,
                      const int32_t *dst_pages, int32_t n, hipStream_t stream);

/* Consumer stand-in for the layered load (not in the paper: it stands in
 * for the attention over layer `layer` that a layered restore lets start
 * early).  For each i < n, d_out[i] (device uint64, out_capacity >= n
 * entries, 8-byte aligned) = the XOR of the little-endian 64-bit words of
 * page pages[i]'s piece of that layer, XOR'd with its 8-byte scale word
 * when the cache has scales.  pages: host int32[n] in [0, P), read before
 * return.  Asynchronous on `stream`, which may wait on a layer_done event
 * of ea_load_blocks_layered first. */
int ea_layer_checksum(ea_cache *cache, int32_t layer, const int32_t *pages,
                      int32_t n, uint64_t *d_out, int64_t out_capacity,
                      hipStream_t stream);

/* How stores and loads cross the host link:
 *  EA_PLAN_DIRECT: one kernel reads/writes the mapped pinned slots;
 *  EA_PLAN_STAGED: gather/scatter through an HBM staging buffer plus DMA
 *                  copies (hipMemcpyAsync) of runs of consecutive slots;
 *  EA_PLAN_AUTO:   the library's measured default per direction.
 * The environment variable EA_TRANSFER=direct|staged overrides AUTO. */
enum { EA_PLAN_AUTO = 0, EA_PLAN_DIRECT = 1, EA_PLAN_STAGED = 2 };
enum { EA_DIR_STORE = 0, EA_DIR_LOAD = 1, EA_DIR_BOTH = 2 };
int ea_tier_set_plan(ea_tier *tier, int direction, int plan);
int ea_tier_get_plan(const ea_tier *tier, int direction, int *plan);

/* Pinned-copy peak of the host link (not in the paper, which quotes the
 * nominal PCIe rate per direction, App. "Offload Cost and Prefix-Survival
 * Model"; here it is the denominator of the host-link fractions): hipMemcpyAsync of `bytes` contiguous
 * bytes between d_buf (device, >= bytes; for EA_DIR_BOTH >= 2*bytes) and the
 * tier's pinned memory, best of `reps`, in GB/s (1e9 bytes/s).  direction:
 * EA_DIR_STORE (device to host), EA_DIR_LOAD (host to device) or EA_DIR_BOTH
 * (both at once on two streams; total bytes over the slower one).  Overwrites
 * the first bytes (2*bytes for BOTH) of the tier's slots, so it returns
 * EA_EINVAL, moving nothing, while any slot in that range is allocated or
 * holds a stored chunk: use it on a tier that holds nothing yet.  The device
 * buffer and the repetition count come from the caller, so the probe
 * allocates nothing and its cost is the caller's choice. */
int ea_peak_probe(ea_tier *tier, void *d_buf, int64_t bytes, int direction,
                  int reps, double *gbps);

/* ------------------------------------------- reuse-distance capacity tool
 *
 * Host-only analysis of a chunk reference stream for sizing the host tier
 * (section 3.2, Eq. 4, the stack-distance principle; App. "Prefix coverage
 * from a reference stream").  No GPU work, no tier needed.  A stream lists
 * 32-byte chunk keys in reference order; in the paper's reference model
 * every request references the full chunks of its prompt, in order, at its
 * first prefix lookup.
 *
 * ea_reuse_distances: prev_dist[i] = the number of distinct chunks other
 * than refs[i] referenced strictly between the previous reference to the
 * same chunk and reference i (the reuse distance D of Eq. 4), or -1 for a
 * first reference; next_dist[i] = the same count from i to the next
 * reference of the chunk, or -1 if there is none.  Either output may be
 * NULL; n may be 0.  O(n log n) time, 40 n bytes of temporary memory.
 *
 * In an LRU tier of K chunks that admits every miss (App. "Reference
 * model"), reference i hits exactly when 0 <= prev_dist[i] < K, for every K
 * at once (Lemma 1 with nothing declined).
 *
 * ea_prefix_coverage: requests j = 0..n_req-1 own the references
 * req_off[j] .. req_off[j+1]-1 (req_off[0] >= 0, non-decreasing, n_req+1
 * entries).  For each capacity caps[c] >= 0 (in chunks),
 * coverage[j*n_caps + c] = the number of leading references of request j
 * that hit in such a tier: its consecutive-prefix host coverage H_j in
 * chunks.  prev_dist comes from ea_reuse_distances over the same stream. */
int ea_reuse_distances(const uint8_t *refs, int64_t n, int64_t *prev_dist,
                       int64_t *next_dist);
int ea_prefix_coverage(const int64_t *prev_dist, const int64_t *req_off,
                       int64_t n_req, const int64_t *caps, int64_t n_caps,
                       int64_t *coverage);

/* The same reference model for one capacity with some misses declined
 * (App. "Reference model"; the setting of Proposition 1): reference i hits
 * if refs[i] is resident and then becomes most recent; a miss with
 * declined[i] != 0 changes nothing; any other miss inserts refs[i] as most
 * recent, first evicting the least-recent chunk when `capacity` chunks are
 * resident.  declined may be NULL (full admission).  hits[i] = 1 for a hit,
 * else 0.  O(n) expected time, O(capacity) memory. */
int ea_lru_simulate(const uint8_t *refs, int64_t n, const uint8_t *declined,
                    int64_t capacity, uint8_t *hits);

/* The host tier's own recency order (App. "Recency order of the host
 * tier"; unlike the reference model, only the leading run of hits is
 * promoted), request by request, for one capacity: request j (refs
 * req_off[j] .. req_off[j+1]-1, req_off[0] = 0) promotes its leading
 * resident chunks, hit_blocks[j] of them; unless declined[j] != 0 it then
 * inserts every later chunk that is absent at that moment, in order
 * (copy-time deduplication, section 4); an insertion into a full tier
 * evicts the least-recent chunk that the request has not promoted or
 * inserted itself (those stay pinned until it ends) and is skipped when
 * there is none.  This is the order ea_tier_lookup / ea_admission_fill /
 * ea_tier_alloc / ea_tier_unpin maintain when every request releases its
 * pins before the next one.  declined may be NULL. */
int ea_lru_simulate_prefix(const uint8_t *refs, const int64_t *req_off,
                           int64_t n_req, const uint8_t *declined,
                           int64_t capacity, int64_t *hit_blocks);

#ifdef __cplusplus
}
#endif
#endif /* EA_H */
