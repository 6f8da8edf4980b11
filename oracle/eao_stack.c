/*
 * eao_stack.c -- oracle of the LRU reference model (TEST INFRASTRUCTURE ONLY).
 *
 * The paper's appendix (reference model behind Lemma 1 and Proposition 1)
 * fixes a stream of chunk references x_1..x_T and an LRU tier of K_H chunks
 * that starts empty.  Reference i hits if x_i is resident and then moves
 * x_i to the most-recent end.  Otherwise it misses; an admitted miss inserts
 * x_i at the most-recent end, evicting the least-recent chunk first when K_H
 * chunks are resident, and a declined miss leaves the tier as it was.  Full
 * admission declines nothing.  Host prefix coverage of a request (the
 * appendix's prefix-coverage model) is the run of hits from its first chunk.
 *
 * This file simulates that model literally, one capacity per call: a
 * chained hash table from key to node and a doubly linked recency list over
 * at most K_H nodes.  O(T) per capacity.
 */
#include <stdlib.h>
#include <string.h>

#include "eao.h"

typedef struct {
  uint8_t key[32];
  int64_t newer, older;  /* recency list; -1 at the ends */
  int64_t chain;         /* next node in the same hash bucket, or -1 */
} lru_node;

typedef struct {
  lru_node *node;
  int64_t *bucket;  /* head node per bucket, or -1 */
  uint64_t mask;
  int64_t used, cap;
  int64_t most, least;  /* most-recent and least-recent node, or -1 */
} lru_model;

static uint64_t key_bucket(const uint8_t *k, uint64_t mask) {
  /* FNV-1a over the whole key */
  uint64_t h = 1469598103934665603ull;
  for (int i = 0; i < 32; ++i) h = (h ^ k[i]) * 1099511628211ull;
  return h & mask;
}

static int64_t find(const lru_model *m, const uint8_t *k) {
  for (int64_t i = m->bucket[key_bucket(k, m->mask)]; i >= 0; i = m->node[i].chain)
    if (memcmp(m->node[i].key, k, 32) == 0) return i;
  return -1;
}

static void unlink_recency(lru_model *m, int64_t i) {
  lru_node *x = &m->node[i];
  if (x->newer >= 0) m->node[x->newer].older = x->older; else m->most = x->older;
  if (x->older >= 0) m->node[x->older].newer = x->newer; else m->least = x->newer;
  x->newer = x->older = -1;
}

static void push_most_recent(lru_model *m, int64_t i) {
  lru_node *x = &m->node[i];
  x->older = m->most;
  x->newer = -1;
  if (m->most >= 0) m->node[m->most].newer = i;
  m->most = i;
  if (m->least < 0) m->least = i;
}

static void unhash(lru_model *m, int64_t i) {
  int64_t *p = &m->bucket[key_bucket(m->node[i].key, m->mask)];
  while (*p != i) p = &m->node[*p].chain;
  *p = m->node[i].chain;
  m->node[i].chain = -1;
}

static void hash_in(lru_model *m, int64_t i) {
  int64_t *head = &m->bucket[key_bucket(m->node[i].key, m->mask)];
  m->node[i].chain = *head;
  *head = i;
}

int eao_lru_reference(const uint8_t *refs, int64_t n, const uint8_t *declined,
                      int64_t capacity, uint8_t *hit_out) {
  if (n < 0 || capacity < 0 || (n > 0 && (refs == NULL || hit_out == NULL)))
    return EAO_EINVAL;
  if (capacity == 0) {  /* nothing is ever resident */
    for (int64_t i = 0; i < n; ++i) hit_out[i] = 0;
    return EAO_OK;
  }
  lru_model m;
  const int64_t cap = capacity < n ? capacity : (n > 0 ? n : 1);
  uint64_t nb = 1;
  while (nb < (uint64_t)cap * 2) nb <<= 1;
  m.node = (lru_node *)malloc(sizeof(lru_node) * (size_t)cap);
  m.bucket = (int64_t *)malloc(sizeof(int64_t) * (size_t)nb);
  if (m.node == NULL || m.bucket == NULL) {
    free(m.node);
    free(m.bucket);
    return EAO_ENOMEM;
  }
  for (uint64_t b = 0; b < nb; ++b) m.bucket[b] = -1;
  m.mask = nb - 1;
  m.used = 0;
  m.cap = cap;
  m.most = m.least = -1;

  for (int64_t i = 0; i < n; ++i) {
    const uint8_t *k = refs + 32 * i;
    const int64_t at = find(&m, k);
    if (at >= 0) {  /* hit: move to the most-recent end */
      hit_out[i] = 1;
      unlink_recency(&m, at);
      push_most_recent(&m, at);
      continue;
    }
    hit_out[i] = 0;
    if (declined != NULL && declined[i]) continue;  /* declined miss */
    int64_t slot;
    if (m.used < capacity && m.used < m.cap) {
      slot = m.used++;
    } else {  /* full: evict the least-recent chunk */
      slot = m.least;
      unlink_recency(&m, slot);
      unhash(&m, slot);
    }
    memcpy(m.node[slot].key, k, 32);
    m.node[slot].newer = m.node[slot].older = -1;
    hash_in(&m, slot);
    push_most_recent(&m, slot);
  }
  free(m.node);
  free(m.bucket);
  return EAO_OK;
}

/* The host tier's own recency order (App. "Recency order of the host tier";
 * the admission rule of section 4 with copy-time deduplication), request by
 * request.  Request j owns refs[req_off[j] .. req_off[j+1]-1]:
 *   1. lookup: its leading resident chunks are promoted in order; the first
 *      absent chunk ends the lookup, and h_out[j] is the number promoted;
 *   2. unless declined[j], every later chunk that is absent at that moment
 *      is inserted in order at the most-recent end (resident ones keep
 *      their place);
 *   3. an insertion into a full tier evicts the least-recent chunk that
 *      this request has not promoted or inserted (those are pinned until
 *      the request ends); with none left the chunk is not inserted. */
int eao_lru_prefix_model(const uint8_t *refs, const int64_t *req_off, int64_t n_req,
                         const uint8_t *declined, int64_t capacity, int64_t *h_out) {
  if (n_req < 0 || capacity < 0 || req_off == NULL || (n_req > 0 && h_out == NULL))
    return EAO_EINVAL;
  if (req_off[0] != 0) return EAO_EINVAL;
  for (int64_t j = 0; j < n_req; ++j)
    if (req_off[j + 1] < req_off[j]) return EAO_EINVAL;
  const int64_t n = req_off[n_req];
  if (n > 0 && refs == NULL) return EAO_EINVAL;
  int64_t longest = 0;
  for (int64_t j = 0; j < n_req; ++j)
    if (req_off[j + 1] - req_off[j] > longest) longest = req_off[j + 1] - req_off[j];
  lru_model m;
  const int64_t cap = capacity < n ? capacity : (n > 0 ? n : 1);
  uint64_t nb = 1;
  while (nb < (uint64_t)cap * 2) nb <<= 1;
  m.node = (lru_node *)malloc(sizeof(lru_node) * (size_t)cap);
  m.bucket = (int64_t *)malloc(sizeof(int64_t) * (size_t)nb);
  int64_t *stamp = (int64_t *)malloc(sizeof(int64_t) * (size_t)cap);  /* request that pinned it */
  uint8_t *insert = (uint8_t *)malloc((size_t)(longest > 0 ? longest : 1));
  if (m.node == NULL || m.bucket == NULL || stamp == NULL || insert == NULL) {
    free(m.node); free(m.bucket); free(stamp); free(insert);
    return EAO_ENOMEM;
  }
  for (uint64_t b = 0; b < nb; ++b) m.bucket[b] = -1;
  for (int64_t i = 0; i < cap; ++i) stamp[i] = -1;
  m.mask = nb - 1;
  m.used = 0;
  m.cap = cap;
  m.most = m.least = -1;

  for (int64_t j = 0; j < n_req; ++j) {
    const int64_t b = req_off[j], len = req_off[j + 1] - b;
    int64_t h = 0;
    if (capacity > 0) {
      while (h < len) {
        const int64_t at = find(&m, refs + 32 * (b + h));
        if (at < 0) break;
        unlink_recency(&m, at);
        push_most_recent(&m, at);
        stamp[at] = j;
        ++h;
      }
    }
    h_out[j] = h;
    if (capacity == 0 || (declined != NULL && declined[j])) continue;
    /* deduplication: decide every insertion before any of them */
    for (int64_t i = h; i < len; ++i) insert[i] = find(&m, refs + 32 * (b + i)) < 0;
    for (int64_t i = h; i < len; ++i) {
      if (!insert[i]) continue;
      const uint8_t *k = refs + 32 * (b + i);
      if (find(&m, k) >= 0) continue;  /* a repeat of a key inserted just now */
      int64_t slot;
      if (m.used < capacity && m.used < m.cap) {
        slot = m.used++;
      } else {
        slot = m.least;
        while (slot >= 0 && stamp[slot] == j) slot = m.node[slot].newer;
        if (slot < 0) continue;  /* every resident chunk is pinned */
        unlink_recency(&m, slot);
        unhash(&m, slot);
      }
      memcpy(m.node[slot].key, k, 32);
      m.node[slot].newer = m.node[slot].older = -1;
      hash_in(&m, slot);
      push_most_recent(&m, slot);
      stamp[slot] = j;
    }
  }
  free(m.node);
  free(m.bucket);
  free(stamp);
  free(insert);
  return EAO_OK;
}
