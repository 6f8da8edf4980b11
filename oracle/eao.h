/*
 * eao.h -- CPU oracle for the KV-offload data path (TEST INFRASTRUCTURE ONLY).
 *
 * This library is the plain, slow, single-threaded definition of what the
 * offload path computes, written from "EfficientAgent: What Makes KV Cache
 * Offloading Work for Concurrent Agents?" (arXiv 2609.33762).  It exists so the
 * tests can check the GPU library bit for bit.  Only the test suite, the smoke
 * check and the CPU-baseline leg of the benchmark may load it; the product
 * path never does.  It shares no code, header, table or constant with the GPU
 * library: the SHA-256 round constants and initial hash value are derived here
 * from their definition (FIPS 180-4, 4.2.2 and 5.3.3) at run time.
 *
 * Everything is host memory.  The "GPU cache" is a host byte array with the
 * same logical layout the GPU library uses:
 *
 *   cache  : [L][P][2][T][H][D] elements of elem_bytes  (one (layer, page)
 *            "piece" of 2*T*H*D*elem_bytes bytes is contiguous)
 *   scales : optional [L][P][2] float32 (K scale, V scale), copied as bytes
 *   tier   : [S][slot_bytes]; a slot holds one chunk of C = chunk_pages
 *            pages (C = 1: one page) of every layer, [L][C][2][T][H][D]
 *            bytes (so one layer of a chunk is contiguous), followed (when
 *            scales exist) by an [L][C][2] float32 trailer padded with
 *            zeros to a multiple of 256 bytes (a store writes the padding
 *            too, so a stored slot is a complete image).
 *
 * Status codes mirror the product library: 0 ok, negative on error, and on
 * error nothing is written.
 *
 * What pins each part (tests/test_oracle_*.py, tests/test_stack_tool.py):
 * SHA-256 by the FIPS 180-4 example values and by hashlib on every block's
 * serialised message; the key chain by the invariants of section 3.2 (equal
 * prefixes, rekeying after an edit, partial tails, continuation from a
 * parent); copies by round trips, untouched bytes, fp8 NaN patterns and numpy
 * restatements of the layout; the tier by a brute-force model, Lemma 1 and
 * Proposition 1 on random streams, the Eq. 6 truth table with its endpoints
 * and the paper's closed forms (footprints, working sets, K_H); the
 * restore cost and OBR of Eq. 2 by the paper's H20 numbers (0.86 us per
 * token, a 5.6 us prefill bound, OBR above 0.84) and the definition's
 * limits; the reference models by brute-force distinct counts and the
 * round-robin closed form.  Parity unpinned: byte compatibility of the keys with LMCache or
 * vLLM, which this definition does not claim.
 */
#ifndef EAO_H
#define EAO_H

#include <stdint.h>
#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  EAO_OK = 0,
  EAO_EINVAL = -1,
  EAO_ENOMEM = -2,
  EAO_ENOSPC = -3,
  EAO_ENOTSUP = -5
};

/* ---------------------------------------------------------------- SHA-256 */

/* SHA-256 of an arbitrary byte string, FIPS 180-4 sections 5.1.1 (padding),
 * 5.2.1 (parsing), 6.2.2 (hash computation). */
void eao_sha256(const uint8_t *msg, uint64_t len, uint8_t digest[32]);

/* The 64 round constants K and the initial hash value H(0), computed from
 * their definition: first 32 bits of the fractional parts of the cube roots
 * of the first 64 primes (4.2.2) and of the square roots of the first 8
 * primes (5.3.3). */
void eao_sha256_constants(uint32_t k[64], uint32_t h0[8]);

/* ------------------------------------------------------ footprint (Eq. 1) */

/* KV bytes per token on one tensor-parallel rank,
 * beta_rank = 2 * L * d * s * max(1, ceil(H_kv / TP))  (section 2, Eq. 1). */
int64_t eao_beta_rank(int64_t layers, int64_t head_dim, int64_t elem_bytes,
                      int64_t kv_heads, int64_t tp);

/* Reuse working-set scale C_reuse = (A - 1) * Nbar * beta_rank in bytes
 * (section 3.2, Eq. 5). */
double eao_working_set_bytes(double active_pool, double mean_prompt_tokens,
                             double beta_rank);

/* Host tier capacity in chunks, K_H = floor(C_H / (b * beta_rank))
 * (section 4, "Which writes a tier can decline"; survival bound of Eq. 4). */
int64_t eao_tier_chunks(int64_t capacity_bytes, int64_t block_tokens,
                        int64_t beta_rank);

/* ------------------------------------------- restore versus recompute (Eq. 2) */

/* Time to restore a prefix of n tokens from the host tier,
 * T_load(n) = n * beta_rank / B_eff + tau_load, in the units of tau_load
 * and of beta_rank / B_eff (section 3.1, Eq. 2). */
double eao_restore_time(double n, double beta_rank, double b_eff, double tau_load);

/* Offload Benefit Ratio OBR(n) = 1 - T_load(n) / T_rec(n) with
 * T_rec(n) = n * t_pf (section 3.1, Eq. 2). */
double eao_obr(double n, double beta_rank, double b_eff, double tau_load, double t_pf);

/* Its limit for long prefixes, where tau_load is amortized:
 * 1 - beta_rank / (B_eff * t_pf) (App. "Offload Cost and Prefix-Survival
 * Model", the per-token cost t_load(n) = beta_rank / B_eff + tau_load / n). */
double eao_obr_limit(double beta_rank, double b_eff, double t_pf);

/* ------------------------------------------------------------------ layout */

typedef struct {
  int32_t num_pages;    /* P: pages in the GPU cache                        */
  int32_t num_layers;   /* L                                                 */
  int32_t page_tokens;  /* T: tokens per page (= hash block size b)          */
  int32_t num_kv_heads; /* H: KV heads held by this rank                     */
  int32_t head_dim;     /* D                                                 */
  int32_t elem_bytes;   /* s: bytes per element (2 for bf16, 1 for fp8)      */
  int32_t has_scales;   /* 1 when a [L][P][2] float32 scale plane exists     */
  int32_t chunk_pages;  /* C: pages per host slot, one key each (>= 1; the
                           paper's 1,024-token host chunk is 64 pages of 16) */
} eao_shape;

int64_t eao_piece_bytes(const eao_shape *sh);  /* 2*T*H*D*s                 */
int64_t eao_page_bytes(const eao_shape *sh);   /* L * piece                 */
int64_t eao_payload_bytes(const eao_shape *sh);/* C * L * piece: slot data  */
int64_t eao_trailer_bytes(const eao_shape *sh);/* L*C*2*4 rounded up to 256, or 0 */
int64_t eao_slot_bytes(const eao_shape *sh);   /* payload + trailer         */
int64_t eao_cache_bytes(const eao_shape *sh);  /* L * P * piece             */
int64_t eao_scale_bytes(const eao_shape *sh);  /* L * P * 8, or 0           */

/* ------------------------------------------------------- chained hashing */

/* Chained prefix-block keys (section 2 "Exact-prefix reuse"; section 3.2:
 * each full chunk's key depends on its entire prefix).
 *
 * Sequence s is tokens[seq_offsets[s] .. seq_offsets[s+1]).  With
 * b = block_tokens and key_{-1} = parents[s] (32 zero bytes when parents is
 * NULL), for every FULL block i:
 *     key_i = SHA-256( LE32(tok[i*b]) || ... || LE32(tok[i*b+b-1]) || key_{i-1} )
 * A trailing partial block gets no key.  Keys of sequence s are written to
 * keys_out[key_offsets_out[s] ..], key_offsets_out has n_seqs+1 entries and
 * key_offsets_out[0] = 0.  A token is hashed as the little-endian bytes of
 * its 32-bit two's-complement value; b >= 1. */
int eao_hash_blocks(const int32_t *tokens, const int64_t *seq_offsets,
                    int32_t n_seqs, int32_t block_tokens,
                    const uint8_t *parents, uint8_t *keys_out,
                    int64_t *key_offsets_out);

/* ------------------------------------------------------------------ copies */

/* Store (host write, "KV copied from GPU to host", section 2): for every i
 * with mask[i] != 0 (mask NULL = all), slot host_slots[i] receives pages
 * block_ids[i*C .. i*C+C-1] of every layer (K and V), page i*C+c at chunk
 * position c, and, with scales, their scales plus zero padding as the slot
 * trailer.  Nothing else changes.  Admitted slots must be distinct; ids
 * and slots must be in range.  n counts slots (block_ids has n*C entries). */
int eao_store_blocks(const eao_shape *sh, const uint8_t *cache,
                     const uint8_t *scales, uint8_t *tier, int64_t num_slots,
                     const int32_t *block_ids, const int64_t *host_slots,
                     const uint8_t *mask, int32_t n);

/* Load (host restore, section 3.1): pages dst_pages[i*C .. i*C+C-1] of
 * every layer receive the chunk in slot host_slots[i], chunk position c
 * into page dst_pages[i*C+c] (with its scales).  The n*C destination pages
 * must be distinct. */
int eao_load_blocks(const eao_shape *sh, const uint8_t *tier,
                    int64_t num_slots, uint8_t *cache, uint8_t *scales,
                    const int64_t *host_slots, const int32_t *dst_pages,
                    int32_t n);

/* The part of the load that touches one layer: after it has run for every
 * layer the state equals eao_load_blocks'. */
int eao_load_layer(const eao_shape *sh, const uint8_t *tier,
                   int64_t num_slots, uint8_t *cache, uint8_t *scales,
                   const int64_t *host_slots, const int32_t *dst_pages,
                   int32_t n, int32_t layer);

/* Consumer stand-in of the layered load (not in the paper): out[i] = XOR
 * of the little-endian 64-bit words of page pages[i]'s piece of `layer`,
 * XOR'd with its 8-byte scale word when the shape has scales. */
int eao_layer_checksum(const eao_shape *sh, const uint8_t *cache,
                       const uint8_t *scales, int32_t layer,
                       const int32_t *pages, int32_t n, uint64_t *out);

/* ---------------------------------------------------- host tier metadata */

/* Slot states. */
enum { EAO_SLOT_FREE = 0, EAO_SLOT_PENDING = 1, EAO_SLOT_RESIDENT = 2 };

/* Admission modes: the conditioned rule of Eq. 6 and its two endpoints
 * (section 4: offload without admission is p = 0, fixed admission p = 1). */
enum { EAO_ADMIT_CONDITIONED = 0, EAO_ADMIT_ALWAYS = 1, EAO_ADMIT_FIXED = 2 };

typedef struct {
  int64_t theta_ppm;        /* occupancy threshold in parts per million
                               (950000 = 0.95); full when
                               registered * 1e6 >= theta_ppm * K_H            */
  int64_t kappa;            /* write threshold in full blocks                 */
  int64_t block_tokens;     /* b                                              */
  int64_t beta_rank;        /* bytes per token per rank for C_reuse           */
  int64_t activity_window;  /* window for A_t and e_t, in caller clock units:
                               an event at time t counts when t > now - W     */
  int32_t length_window;    /* N_t = mean of the last this-many first lookups */
  int32_t mode;             /* EAO_ADMIT_*                                    */
  int32_t telemetry;        /* 1: the tier's state is a fresh report;
                               0: no report, the estimate alone decides       */
  int32_t _pad;
} eao_policy;

typedef struct {
  int64_t n_tokens;  /* n: prompt tokens                                      */
  int64_t h_tokens;  /* h: prompt tokens the host tier already holds          */
  int64_t task_id;   /* agent/task identity for A_t                           */
  int64_t now;       /* caller clock (e.g. microseconds or turns), never
                        smaller than the previous request's                   */
  int32_t decided;   /* -1: first lookup, decide now; 0/1: keep earlier save  */
  int32_t _pad;
} eao_request;

typedef struct {
  int64_t capacity_slots;   /* K_H                                            */
  int64_t allocated;        /* slots holding a key: pending + resident        */
  int64_t registered;       /* resident chunks (store issued): the occupancy
                               o_t = registered / K_H of Eq. 10               */
  int64_t pinned;           /* slots with a pin count > 0                     */
  int64_t evictions_total;  /* evictions made to allocate                     */
  int64_t evictions_window; /* of those, within the activity window at clock  */
  int64_t clock;            /* last request clock                             */
  int64_t active_tasks;     /* A_t at the last decision                       */
  double  mean_prompt;      /* N_t at the last decision (display only)        */
  double  working_set;      /* C_reuse at the last decision (display only)    */
  int32_t last_pressure;    /* p_t at the last decision                       */
  int32_t last_save;
} eao_tier_stats;

typedef struct eao_tier eao_tier;

/* K_H = floor(capacity_bytes / slot_bytes); fails with EAO_EINVAL if K_H < 1.
 * capacity_bytes is also the C_H that the admission rule compares the
 * working-set estimate with. */
int eao_tier_create(const eao_shape *sh, int64_t capacity_bytes,
                    eao_tier **out);
int eao_tier_destroy(eao_tier *t);
int64_t eao_tier_capacity(const eao_tier *t);

/* Consecutive-prefix lookup (section 3.2; App. "Prefix coverage"): the hit
 * count is the largest k with key_0..key_{k-1} all resident; a lookup stops
 * at the first absent key, and a key whose slot is still PENDING (allocated,
 * store not yet issued) counts as absent.  Hits are moved to the most-recent end in
 * increasing position order and pinned (one pin each).  slots_out[i] for
 * i < hit count gets the slot. */
int eao_tier_lookup(eao_tier *t, const uint8_t *keys, int64_t n,
                    int64_t *hit_blocks, int64_t *slots_out);

/* Write admission (section 4, Eq. 6; App. "Runtime Admission Details",
 * Eq. 10) plus copy-time deduplication: save_out gets save(r), and
 * mask_out[i] = save && the tier holds no slot under key_i (pending or
 * resident: deduplication also sees allocations whose store is not issued). */
int eao_admission_fill(eao_tier *t, const eao_policy *p, const eao_request *r,
                       const uint8_t *keys, int64_t n_keys, uint8_t *mask_out,
                       int32_t *save_out);

/* Telemetry a worker publishes (App. "Runtime Admission Details": every
 * second, the chunks registered in the tier, its capacity K_H and the
 * evictions made to allocate in the last window). */
typedef struct {
  int64_t time;            /* clock value the report was taken at           */
  int64_t registered;      /* resident chunks (store issued); a pending
                              allocation is not registered yet             */
  int64_t capacity_slots;  /* K_H                                           */
  int64_t evictions;       /* e_t: evictions stamped in (time - window, time] */
} eao_tier_report;

/* Take the report at time `now` (not below the tier's clock) and advance
 * the tier's clock to it: evictions are stamped with the tier's clock, the
 * latest time it has been told by a decision or a report. */
int eao_tier_publish(eao_tier *t, int64_t now, int64_t window, eao_tier_report *out);

/* eao_admission_fill with the "full and evicting" factor taken from the
 * scheduler's copy of a published report: used when policy->telemetry is 1,
 * report is not NULL and 0 <= r->now - report->time <= max_age (a fresh
 * report); otherwise the working-set estimate alone decides (Eq. 10 and the
 * text after it).  max_age >= 0. */
int eao_admission_fill_report(eao_tier *t, const eao_policy *p, const eao_request *r,
                              const eao_tier_report *report, int64_t max_age,
                              const uint8_t *keys, int64_t n_keys, uint8_t *mask_out,
                              int32_t *save_out);

/* Allocate a slot for every i with mask[i] != 0 whose key the tier does not
 * hold yet (pending or resident): the lowest-numbered free slot, else the
 * least-recent resident unpinned slot (an eviction).  New slots are PENDING
 * under the key, placed at the most-recent end in increasing position order,
 * and pinned; they count as registered (occupancy) only once their store is
 * issued (eao_tier_mark_stored).  slots_out[i] = -1 where nothing was allocated; once no victim is
 * left, every later admitted block gets -1.  *allocated gets the count. */
int eao_tier_alloc(eao_tier *t, const uint8_t *keys, const uint8_t *mask,
                   int64_t n, int64_t *slots_out, int64_t *allocated);

/* Metadata effect of a store issued to these slots: PENDING slots become
 * RESIDENT (entries with mask 0 are skipped; mask NULL = all). */
int eao_tier_mark_stored(eao_tier *t, const int64_t *slots,
                         const uint8_t *mask, int64_t n);

/* Drop one pin from each slot; a PENDING slot whose last pin goes away is
 * abandoned: its key is dropped and the slot becomes free. */
int eao_tier_unpin(eao_tier *t, const int64_t *slots, int64_t n);

int eao_tier_stats_get(const eao_tier *t, eao_tier_stats *s);

/* Full metadata image for bit-exact comparison: for every slot its state,
 * pin count and key (zeros when free), and the resident/pending slots from
 * least-recent to most-recent in lru_out (*n_lru entries). */
int eao_tier_export(const eao_tier *t, uint8_t *state_out, int32_t *pins_out,
                    uint8_t *keys_out, int64_t *lru_out, int64_t *n_lru);


/* ------------------------------------------------- LRU reference model */

/* The appendix's LRU reference model (behind Equation (4), Lemma 1 and
 * Proposition 1), simulated for one capacity.  refs holds n 32-byte chunk
 * keys in reference order; declined (n bytes, NULL = full admission) marks
 * references whose miss is declined.  The tier of `capacity` chunks starts
 * empty.  hit_out[i] = 1 if reference i finds its chunk resident (and
 * promotes it to the most-recent end), else 0 (an admitted miss inserts the
 * chunk at the most-recent end, evicting the least-recent one if the tier
 * is full; a declined miss changes nothing). */
int eao_lru_reference(const uint8_t *refs, int64_t n, const uint8_t *declined,
                      int64_t capacity, uint8_t *hit_out);

/* The host tier's own order, request by request (App. "Recency order of
 * the host tier"; section 4, Eq. 6 and copy-time deduplication): request j
 * (refs[req_off[j] .. req_off[j+1]-1], req_off[0] = 0) promotes its leading
 * resident chunks (h_out[j] of them, the lookup's hits); unless declined[j]
 * it then inserts, in order, each later chunk absent at that moment; an
 * insertion into a full tier evicts the least-recent chunk the request has
 * not itself promoted or inserted, and is skipped if there is none.
 * declined may be NULL (every request admitted). */
int eao_lru_prefix_model(const uint8_t *refs, const int64_t *req_off, int64_t n_req,
                         const uint8_t *declined, int64_t capacity, int64_t *h_out);

#ifdef __cplusplus
}
#endif
#endif /* EAO_H */
