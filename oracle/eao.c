/*
 * eao.c -- CPU oracle: SHA-256, chained block keys, layout sizes, copies.
 * TEST INFRASTRUCTURE ONLY (see eao.h).  Plain single-threaded C; nothing
 * here is blocked, fused or reordered beyond what the definitions state.
 */
#include "eao.h"

#include <stdlib.h>
#include <string.h>

/* ================================================================ SHA-256 */
/* FIPS 180-4.  Section numbers below are the standard's. */

static int is_prime(unsigned p) {
  if (p < 2) return 0;
  for (unsigned d = 2; d * d <= p; ++d)
    if (p % d == 0) return 0;
  return 1;
}

/* largest x with x*x <= v */
static unsigned __int128 isqrt128(unsigned __int128 v) {
  unsigned __int128 lo = 0, hi = ((unsigned __int128)1) << 64;
  while (lo < hi) {
    unsigned __int128 mid = lo + (hi - lo + 1) / 2;
    if (mid * mid <= v) lo = mid; else hi = mid - 1;
  }
  return lo;
}

/* largest x with x*x*x <= v (v < 2^120 here, so x < 2^40) */
static unsigned __int128 icbrt128(unsigned __int128 v) {
  unsigned __int128 lo = 0, hi = ((unsigned __int128)1) << 40;
  while (lo < hi) {
    unsigned __int128 mid = lo + (hi - lo + 1) / 2;
    if (mid * mid * mid <= v) lo = mid; else hi = mid - 1;
  }
  return lo;
}

/* 4.2.2: K_t = first 32 bits of the fractional part of cbrt(p_t);
 * 5.3.3: H(0)_j = first 32 bits of the fractional part of sqrt(p_j).
 * floor(frac(r) * 2^32) = floor(r * 2^32) mod 2^32, and r * 2^32 is the
 * integer cube (square) root of p * 2^96 (p * 2^64). */
void eao_sha256_constants(uint32_t k[64], uint32_t h0[8]) {
  unsigned found = 0;
  for (unsigned p = 2; found < 64; ++p) {
    if (!is_prime(p)) continue;
    unsigned __int128 c = icbrt128(((unsigned __int128)p) << 96);
    k[found] = (uint32_t)(c & 0xffffffffu);
    if (found < 8) {
      unsigned __int128 s = isqrt128(((unsigned __int128)p) << 64);
      h0[found] = (uint32_t)(s & 0xffffffffu);
    }
    ++found;
  }
}

static uint32_t g_k[64], g_h0[8];
static int g_have_constants = 0;

static void ensure_constants(void) {
  if (!g_have_constants) {
    eao_sha256_constants(g_k, g_h0);
    g_have_constants = 1;
  }
}

/* 3.2 / 4.1.2 operations on 32-bit words */
static uint32_t rotr(uint32_t x, unsigned n) { return (x >> n) | (x << (32 - n)); }
static uint32_t ch(uint32_t x, uint32_t y, uint32_t z) { return (x & y) ^ (~x & z); }
static uint32_t maj(uint32_t x, uint32_t y, uint32_t z) { return (x & y) ^ (x & z) ^ (y & z); }
static uint32_t big_sigma0(uint32_t x) { return rotr(x, 2) ^ rotr(x, 13) ^ rotr(x, 22); }
static uint32_t big_sigma1(uint32_t x) { return rotr(x, 6) ^ rotr(x, 11) ^ rotr(x, 25); }
static uint32_t small_sigma0(uint32_t x) { return rotr(x, 7) ^ rotr(x, 18) ^ (x >> 3); }
static uint32_t small_sigma1(uint32_t x) { return rotr(x, 17) ^ rotr(x, 19) ^ (x >> 10); }

/* 6.2.2, steps 1-4, for one 512-bit block M (64 bytes) */
static void sha256_block(uint32_t H[8], const uint8_t M[64]) {
  uint32_t W[64];
  for (int t = 0; t < 16; ++t)  /* 5.2.1: words are big-endian */
    W[t] = ((uint32_t)M[4 * t] << 24) | ((uint32_t)M[4 * t + 1] << 16) |
           ((uint32_t)M[4 * t + 2] << 8) | (uint32_t)M[4 * t + 3];
  for (int t = 16; t < 64; ++t)
    W[t] = small_sigma1(W[t - 2]) + W[t - 7] + small_sigma0(W[t - 15]) + W[t - 16];
  uint32_t a = H[0], b = H[1], c = H[2], d = H[3];
  uint32_t e = H[4], f = H[5], g = H[6], h = H[7];
  for (int t = 0; t < 64; ++t) {
    uint32_t T1 = h + big_sigma1(e) + ch(e, f, g) + g_k[t] + W[t];
    uint32_t T2 = big_sigma0(a) + maj(a, b, c);
    h = g; g = f; f = e; e = d + T1;
    d = c; c = b; b = a; a = T1 + T2;
  }
  H[0] += a; H[1] += b; H[2] += c; H[3] += d;
  H[4] += e; H[5] += f; H[6] += g; H[7] += h;
}

void eao_sha256(const uint8_t *msg, uint64_t len, uint8_t digest[32]) {
  ensure_constants();
  uint32_t H[8];
  for (int j = 0; j < 8; ++j) H[j] = g_h0[j];
  /* 5.1.1 padding: the message, a 1 bit, zeros up to 448 mod 512 bits, and
   * the 64-bit big-endian bit length.  Whole blocks straight from msg. */
  uint64_t full = len / 64;
  for (uint64_t i = 0; i < full; ++i) sha256_block(H, msg + 64 * i);
  uint8_t tail[128];
  memset(tail, 0, sizeof tail);
  uint64_t rem = len - 64 * full;
  if (rem) memcpy(tail, msg + 64 * full, rem);
  tail[rem] = 0x80;
  uint64_t tail_len = (rem + 1 + 8 <= 64) ? 64 : 128;
  uint64_t bits = len * 8;
  for (int i = 0; i < 8; ++i) tail[tail_len - 1 - i] = (uint8_t)(bits >> (8 * i));
  sha256_block(H, tail);
  if (tail_len == 128) sha256_block(H, tail + 64);
  for (int j = 0; j < 8; ++j) {  /* 6.2.2 step 4 output, big-endian */
    digest[4 * j] = (uint8_t)(H[j] >> 24);
    digest[4 * j + 1] = (uint8_t)(H[j] >> 16);
    digest[4 * j + 2] = (uint8_t)(H[j] >> 8);
    digest[4 * j + 3] = (uint8_t)H[j];
  }
}

/* ======================================================= footprint, sizes */

int64_t eao_beta_rank(int64_t layers, int64_t head_dim, int64_t elem_bytes,
                      int64_t kv_heads, int64_t tp) {
  /* Eq. 1: 2 L d s max(1, ceil(H_kv / TP)) */
  int64_t heads = (kv_heads + tp - 1) / tp;
  if (heads < 1) heads = 1;
  return 2 * layers * head_dim * elem_bytes * heads;
}

double eao_working_set_bytes(double active_pool, double mean_prompt_tokens,
                             double beta_rank) {
  /* Eq. 5: (A - 1) Nbar beta_rank */
  return (active_pool - 1.0) * mean_prompt_tokens * beta_rank;
}

int64_t eao_tier_chunks(int64_t capacity_bytes, int64_t block_tokens,
                        int64_t beta_rank) {
  return capacity_bytes / (block_tokens * beta_rank);
}

double eao_restore_time(double n, double beta_rank, double b_eff, double tau_load) {
  /* Eq. 2: T_load(n) = n beta_rank / B_eff + tau_load */
  return n * beta_rank / b_eff + tau_load;
}

double eao_obr(double n, double beta_rank, double b_eff, double tau_load, double t_pf) {
  /* Eq. 2: OBR(n) = 1 - T_load(n) / T_rec(n), T_rec(n) = n t_pf */
  return 1.0 - eao_restore_time(n, beta_rank, b_eff, tau_load) / (n * t_pf);
}

double eao_obr_limit(double beta_rank, double b_eff, double t_pf) {
  /* n -> infinity: tau_load / n vanishes */
  return 1.0 - beta_rank / (b_eff * t_pf);
}

int64_t eao_piece_bytes(const eao_shape *sh) {
  return 2LL * sh->page_tokens * sh->num_kv_heads * sh->head_dim * sh->elem_bytes;
}
int64_t eao_page_bytes(const eao_shape *sh) {
  return (int64_t)sh->num_layers * eao_piece_bytes(sh);
}
int64_t eao_payload_bytes(const eao_shape *sh) {
  return (int64_t)sh->chunk_pages * eao_page_bytes(sh);
}
int64_t eao_trailer_bytes(const eao_shape *sh) {
  if (!sh->has_scales) return 0;
  int64_t raw = (int64_t)sh->num_layers * sh->chunk_pages * 2 * 4;
  return (raw + 255) / 256 * 256;
}
int64_t eao_slot_bytes(const eao_shape *sh) {
  return eao_payload_bytes(sh) + eao_trailer_bytes(sh);
}
int64_t eao_cache_bytes(const eao_shape *sh) {
  return (int64_t)sh->num_layers * sh->num_pages * eao_piece_bytes(sh);
}
int64_t eao_scale_bytes(const eao_shape *sh) {
  return sh->has_scales ? (int64_t)sh->num_layers * sh->num_pages * 8 : 0;
}

static int shape_ok(const eao_shape *sh) {
  if (!sh) return 0;
  if (sh->num_pages < 1 || sh->num_layers < 1 || sh->page_tokens < 1 ||
      sh->num_kv_heads < 1 || sh->head_dim < 1 || sh->elem_bytes < 1)
    return 0;
  if (sh->has_scales != 0 && sh->has_scales != 1) return 0;
  if (sh->chunk_pages < 1) return 0;
  return 1;
}

/* ================================================= chained block hashing */

int eao_hash_blocks(const int32_t *tokens, const int64_t *seq_offsets,
                    int32_t n_seqs, int32_t block_tokens,
                    const uint8_t *parents, uint8_t *keys_out,
                    int64_t *key_offsets_out) {
  if (n_seqs < 0 || block_tokens < 1 || !key_offsets_out) return EAO_EINVAL;
  if (n_seqs > 0 && !seq_offsets) return EAO_EINVAL;
  int64_t total_keys = 0;
  for (int32_t s = 0; s < n_seqs; ++s) {
    if (seq_offsets[s] < 0 || seq_offsets[s + 1] < seq_offsets[s]) return EAO_EINVAL;
    total_keys += (seq_offsets[s + 1] - seq_offsets[s]) / block_tokens;
  }
  if (total_keys > 0 && (!tokens || !keys_out)) return EAO_EINVAL;

  uint64_t msg_len = 4ull * (uint64_t)block_tokens + 32;
  uint8_t *msg = (uint8_t *)malloc(msg_len);
  if (!msg) return EAO_ENOMEM;

  int64_t k = 0;
  key_offsets_out[0] = 0;
  for (int32_t s = 0; s < n_seqs; ++s) {
    const int32_t *seq = tokens ? tokens + seq_offsets[s] : NULL;
    int64_t n_full = (seq_offsets[s + 1] - seq_offsets[s]) / block_tokens;
    uint8_t prev[32];
    if (parents) memcpy(prev, parents + 32 * (int64_t)s, 32);
    else memset(prev, 0, 32);
    for (int64_t i = 0; i < n_full; ++i) {
      /* message = LE32 of the block's tokens, then the previous key */
      for (int32_t j = 0; j < block_tokens; ++j) {
        uint32_t v = (uint32_t)seq[i * block_tokens + j];
        msg[4 * j] = (uint8_t)v;
        msg[4 * j + 1] = (uint8_t)(v >> 8);
        msg[4 * j + 2] = (uint8_t)(v >> 16);
        msg[4 * j + 3] = (uint8_t)(v >> 24);
      }
      memcpy(msg + 4 * (uint64_t)block_tokens, prev, 32);
      eao_sha256(msg, msg_len, keys_out + 32 * k);
      memcpy(prev, keys_out + 32 * k, 32);
      ++k;
    }
    key_offsets_out[s + 1] = k;
  }
  free(msg);
  return EAO_OK;
}

/* =================================================================== copies */

int eao_store_blocks(const eao_shape *sh, const uint8_t *cache,
                     const uint8_t *scales, uint8_t *tier, int64_t num_slots,
                     const int32_t *block_ids, const int64_t *host_slots,
                     const uint8_t *mask, int32_t n) {
  if (!shape_ok(sh) || n < 0 || num_slots < 0) return EAO_EINVAL;
  if (sh->has_scales != (scales != NULL)) return EAO_EINVAL;
  if (n == 0) return EAO_OK;
  if (!cache || !tier || !block_ids || !host_slots) return EAO_EINVAL;
  /* validate everything before writing anything */
  uint8_t *seen = (uint8_t *)calloc((size_t)(num_slots > 0 ? num_slots : 1), 1);
  if (!seen) return EAO_ENOMEM;
  const int64_t C = sh->chunk_pages;
  for (int32_t i = 0; i < n; ++i) {
    if (mask && !mask[i]) continue;
    int bad = host_slots[i] < 0 || host_slots[i] >= num_slots || seen[host_slots[i]];
    for (int64_t c = 0; c < C && !bad; ++c)
      bad = block_ids[i * C + c] < 0 || block_ids[i * C + c] >= sh->num_pages;
    if (bad) {
      free(seen);
      return EAO_EINVAL;
    }
    seen[host_slots[i]] = 1;
  }
  free(seen);

  const int64_t piece = eao_piece_bytes(sh);
  const int64_t slot_bytes = eao_slot_bytes(sh);
  const int64_t P = sh->num_pages;
  const int64_t L = sh->num_layers;
  for (int32_t i = 0; i < n; ++i) {
    if (mask && !mask[i]) continue;
    uint8_t *slot = tier + host_slots[i] * slot_bytes;
    for (int64_t l = 0; l < L; ++l)
      for (int64_t c = 0; c < C; ++c)  /* chunk position c of layer l */
        memcpy(slot + (l * C + c) * piece,
               cache + (l * P + block_ids[i * C + c]) * piece, (size_t)piece);
    if (sh->has_scales) {
      /* trailer: 8 bytes of scales per (layer, chunk position), then zeros */
      uint8_t *trailer = slot + eao_payload_bytes(sh);
      for (int64_t l = 0; l < L; ++l)
        for (int64_t c = 0; c < C; ++c)
          memcpy(trailer + 8 * (l * C + c), scales + (l * P + block_ids[i * C + c]) * 8, 8);
      memset(trailer + 8 * L * C, 0, (size_t)(eao_trailer_bytes(sh) - 8 * L * C));
    }
  }
  return EAO_OK;
}

static int load_validate(const eao_shape *sh, const uint8_t *tier,
                         int64_t num_slots, uint8_t *cache,
                         const uint8_t *scales, const int64_t *host_slots,
                         const int32_t *dst_pages, int32_t n) {
  if (!shape_ok(sh) || n < 0 || num_slots < 0) return EAO_EINVAL;
  if (sh->has_scales != (scales != NULL)) return EAO_EINVAL;
  if (n == 0) return EAO_OK;
  if (!cache || !tier || !host_slots || !dst_pages) return EAO_EINVAL;
  uint8_t *seen = (uint8_t *)calloc((size_t)sh->num_pages, 1);
  if (!seen) return EAO_ENOMEM;
  const int64_t C = sh->chunk_pages;
  for (int32_t i = 0; i < n; ++i) {
    int bad = host_slots[i] < 0 || host_slots[i] >= num_slots;
    for (int64_t c = 0; c < C && !bad; ++c) {
      const int32_t d = dst_pages[i * C + c];
      bad = d < 0 || d >= sh->num_pages || seen[d];
      if (!bad) seen[d] = 1;
    }
    if (bad) {
      free(seen);
      return EAO_EINVAL;
    }
  }
  free(seen);
  return EAO_OK;
}

static void load_one_layer(const eao_shape *sh, const uint8_t *tier,
                           uint8_t *cache, uint8_t *scales,
                           const int64_t *host_slots, const int32_t *dst_pages,
                           int32_t n, int32_t l) {
  const int64_t piece = eao_piece_bytes(sh);
  const int64_t slot_bytes = eao_slot_bytes(sh);
  const int64_t P = sh->num_pages;
  const int64_t C = sh->chunk_pages;
  for (int32_t i = 0; i < n; ++i) {
    const uint8_t *slot = tier + host_slots[i] * slot_bytes;
    for (int64_t c = 0; c < C; ++c) {
      const int64_t d = dst_pages[i * C + c];
      memcpy(cache + ((int64_t)l * P + d) * piece, slot + ((int64_t)l * C + c) * piece,
             (size_t)piece);
      if (sh->has_scales)
        memcpy(scales + ((int64_t)l * P + d) * 8,
               slot + eao_payload_bytes(sh) + 8 * ((int64_t)l * C + c), 8);
    }
  }
}

int eao_load_blocks(const eao_shape *sh, const uint8_t *tier,
                    int64_t num_slots, uint8_t *cache, uint8_t *scales,
                    const int64_t *host_slots, const int32_t *dst_pages,
                    int32_t n) {
  int rc = load_validate(sh, tier, num_slots, cache, scales, host_slots,
                         dst_pages, n);
  if (rc != EAO_OK || n == 0) return rc;
  for (int32_t l = 0; l < sh->num_layers; ++l)
    load_one_layer(sh, tier, cache, scales, host_slots, dst_pages, n, l);
  return EAO_OK;
}

int eao_load_layer(const eao_shape *sh, const uint8_t *tier,
                   int64_t num_slots, uint8_t *cache, uint8_t *scales,
                   const int64_t *host_slots, const int32_t *dst_pages,
                   int32_t n, int32_t layer) {
  int rc = load_validate(sh, tier, num_slots, cache, scales, host_slots,
                         dst_pages, n);
  if (rc != EAO_OK || n == 0) return rc;
  if (layer < 0 || layer >= sh->num_layers) return EAO_EINVAL;
  load_one_layer(sh, tier, cache, scales, host_slots, dst_pages, n, layer);
  return EAO_OK;
}

/* Consumer stand-in of the layered load: for each listed page, the XOR of
 * the little-endian 64-bit words of its piece of layer `layer`, XOR'd with
 * its 8-byte scale word when the shape has scales.  Not in the paper (it
 * stands in for the attention that reads layer l once it has arrived). */
int eao_layer_checksum(const eao_shape *sh, const uint8_t *cache,
                       const uint8_t *scales, int32_t layer,
                       const int32_t *pages, int32_t n, uint64_t *out) {
  if (!shape_ok(sh) || !cache || n < 0 || (n > 0 && (!pages || !out)))
    return EAO_EINVAL;
  if (layer < 0 || layer >= sh->num_layers) return EAO_EINVAL;
  if (sh->has_scales && !scales) return EAO_EINVAL;
  const int64_t piece = eao_piece_bytes(sh);
  const int64_t P = sh->num_pages;
  for (int32_t i = 0; i < n; ++i)
    if (pages[i] < 0 || pages[i] >= P) return EAO_EINVAL;
  for (int32_t i = 0; i < n; ++i) {
    const uint8_t *p = cache + ((int64_t)layer * P + pages[i]) * piece;
    uint64_t x = 0;
    for (int64_t w = 0; w < piece / 8; ++w) {
      uint64_t v = 0;
      for (int b = 0; b < 8; ++b) v |= (uint64_t)p[8 * w + b] << (8 * b);
      x ^= v;
    }
    if (sh->has_scales) {
      const uint8_t *s = scales + ((int64_t)layer * P + pages[i]) * 8;
      uint64_t v = 0;
      for (int b = 0; b < 8; ++b) v |= (uint64_t)s[b] << (8 * b);
      x ^= v;
    }
    out[i] = x;
  }
  return EAO_OK;
}
