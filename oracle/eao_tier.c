/*
 * eao_tier.c -- CPU oracle: host-tier metadata (key map, LRU recency, pins)
 * and working-set-aware write admission.  TEST INFRASTRUCTURE ONLY.
 *
 * The LRU host tier of App. "Runtime Admission Details" and "Recency order
 * of the host tier": new chunks join at the tail of a recency list; a lookup
 * promotes only its leading hits to the tail; nothing leaves except when an
 * allocation finds no free slot, which then takes the first unpinned
 * resident chunk from the head.
 */
#include "eao.h"

#include <stdlib.h>
#include <string.h>

struct eao_tier {
  int64_t K;              /* K_H slots                                        */
  int64_t capacity_bytes; /* C_H                                              */
  uint8_t *state;         /* [K] EAO_SLOT_*                                   */
  int32_t *pins;          /* [K]                                              */
  uint8_t *keys;          /* [K][32]                                          */
  /* recency: doubly linked list of registered slots, head = least recent */
  int64_t *prev, *next;
  int64_t head, tail;
  /* key -> slot: chained hash buckets over slot indices */
  int64_t nbuckets;
  int64_t *bucket;        /* [nbuckets] first slot or -1                      */
  int64_t *chain;         /* [K] next slot in the same bucket or -1           */
  /* allocated: slots holding a key (pending + resident); registered: chunks
   * whose store has been issued, the numerator of the occupancy o_t (a store
   * allocates its buffers before it registers its chunks) */
  int64_t allocated, registered;
  /* eviction log (clock stamps), only the last stamp and the count matter */
  int64_t evictions_total;
  int64_t *evict_stamp;   /* growing array of stamps                          */
  int64_t evict_cap;
  /* first-lookup log */
  int64_t *log_task, *log_n, *log_time;
  int64_t log_len, log_cap;
  int64_t clock;
  int have_clock;
  int64_t last_window;    /* activity window of the last decision           */
  /* last decision, for stats */
  int64_t last_active;
  double last_mean, last_ws;
  int32_t last_pressure, last_save;
};

/* --------------------------------------------------------------- key map */

static uint64_t key_hash(const uint8_t *k) {
  uint64_t h = 0;
  for (int i = 0; i < 8; ++i) h |= (uint64_t)k[i] << (8 * i);
  return h;
}

static int64_t map_find(const eao_tier *t, const uint8_t *key) {
  int64_t s = t->bucket[key_hash(key) % (uint64_t)t->nbuckets];
  while (s >= 0) {
    if (memcmp(t->keys + 32 * s, key, 32) == 0) return s;
    s = t->chain[s];
  }
  return -1;
}

static void map_insert(eao_tier *t, int64_t slot) {
  uint64_t b = key_hash(t->keys + 32 * slot) % (uint64_t)t->nbuckets;
  t->chain[slot] = t->bucket[b];
  t->bucket[b] = slot;
}

static void map_remove(eao_tier *t, int64_t slot) {
  uint64_t b = key_hash(t->keys + 32 * slot) % (uint64_t)t->nbuckets;
  int64_t *link = &t->bucket[b];
  while (*link != slot) link = &t->chain[*link];
  *link = t->chain[slot];
  t->chain[slot] = -1;
}

/* ---------------------------------------------------------- recency list */

static void lru_unlink(eao_tier *t, int64_t s) {
  if (t->prev[s] >= 0) t->next[t->prev[s]] = t->next[s]; else t->head = t->next[s];
  if (t->next[s] >= 0) t->prev[t->next[s]] = t->prev[s]; else t->tail = t->prev[s];
  t->prev[s] = t->next[s] = -1;
}

static void lru_push_recent(eao_tier *t, int64_t s) {
  t->prev[s] = t->tail;
  t->next[s] = -1;
  if (t->tail >= 0) t->next[t->tail] = s; else t->head = s;
  t->tail = s;
}

/* ------------------------------------------------------------ life cycle */

int eao_tier_create(const eao_shape *sh, int64_t capacity_bytes,
                    eao_tier **out) {
  if (!sh || !out || capacity_bytes <= 0) return EAO_EINVAL;
  int64_t slot_bytes = eao_slot_bytes(sh);
  if (slot_bytes <= 0) return EAO_EINVAL;
  int64_t K = capacity_bytes / slot_bytes;
  if (K < 1) return EAO_EINVAL;
  eao_tier *t = (eao_tier *)calloc(1, sizeof *t);
  if (!t) return EAO_ENOMEM;
  t->K = K;
  t->capacity_bytes = capacity_bytes;
  t->nbuckets = 2 * K + 1;
  t->state = (uint8_t *)calloc((size_t)K, 1);
  t->pins = (int32_t *)calloc((size_t)K, sizeof(int32_t));
  t->keys = (uint8_t *)calloc((size_t)K, 32);
  t->prev = (int64_t *)malloc((size_t)K * sizeof(int64_t));
  t->next = (int64_t *)malloc((size_t)K * sizeof(int64_t));
  t->chain = (int64_t *)malloc((size_t)K * sizeof(int64_t));
  t->bucket = (int64_t *)malloc((size_t)t->nbuckets * sizeof(int64_t));
  if (!t->state || !t->pins || !t->keys || !t->prev || !t->next || !t->chain ||
      !t->bucket) {
    eao_tier_destroy(t);
    return EAO_ENOMEM;
  }
  for (int64_t s = 0; s < K; ++s) t->prev[s] = t->next[s] = t->chain[s] = -1;
  for (int64_t b = 0; b < t->nbuckets; ++b) t->bucket[b] = -1;
  t->head = t->tail = -1;
  *out = t;
  return EAO_OK;
}

int eao_tier_destroy(eao_tier *t) {
  if (!t) return EAO_EINVAL;
  free(t->state); free(t->pins); free(t->keys);
  free(t->prev); free(t->next); free(t->chain); free(t->bucket);
  free(t->evict_stamp);
  free(t->log_task); free(t->log_n); free(t->log_time);
  free(t);
  return EAO_OK;
}

int64_t eao_tier_capacity(const eao_tier *t) { return t ? t->K : -1; }

/* ---------------------------------------------------------------- lookup */

int eao_tier_lookup(eao_tier *t, const uint8_t *keys, int64_t n,
                    int64_t *hit_blocks, int64_t *slots_out) {
  if (!t || n < 0 || !hit_blocks) return EAO_EINVAL;
  if (n > 0 && (!keys || !slots_out)) return EAO_EINVAL;
  int64_t h = 0;
  while (h < n) {
    int64_t s = map_find(t, keys + 32 * h);
    if (s < 0 || t->state[s] != EAO_SLOT_RESIDENT) break;
    slots_out[h] = s;
    ++h;
  }
  /* hits become most recent in increasing position order, and are pinned */
  for (int64_t i = 0; i < h; ++i) {
    lru_unlink(t, slots_out[i]);
    lru_push_recent(t, slots_out[i]);
    t->pins[slots_out[i]] += 1;
  }
  *hit_blocks = h;
  return EAO_OK;
}

/* ------------------------------------------------------------- admission */

static int log_append(eao_tier *t, int64_t task, int64_t n, int64_t now) {
  if (t->log_len == t->log_cap) {
    int64_t cap = t->log_cap ? 2 * t->log_cap : 256;
    int64_t *a = (int64_t *)realloc(t->log_task, (size_t)cap * sizeof(int64_t));
    if (!a) return EAO_ENOMEM;
    t->log_task = a;
    a = (int64_t *)realloc(t->log_n, (size_t)cap * sizeof(int64_t));
    if (!a) return EAO_ENOMEM;
    t->log_n = a;
    a = (int64_t *)realloc(t->log_time, (size_t)cap * sizeof(int64_t));
    if (!a) return EAO_ENOMEM;
    t->log_time = a;
    t->log_cap = cap;
  }
  t->log_task[t->log_len] = task;
  t->log_n[t->log_len] = n;
  t->log_time[t->log_len] = now;
  t->log_len += 1;
  return EAO_OK;
}

/* Where the "tier full and evicting" factor comes from. */
enum { TELEMETRY_POLICY = 0, TELEMETRY_REPORT = 1 };

static int admission(eao_tier *t, const eao_policy *p, const eao_request *r,
                     int source, const eao_tier_report *rep, int64_t max_age,
                     const uint8_t *keys, int64_t n_keys, uint8_t *mask_out,
                     int32_t *save_out) {
  if (!t || !p || !r || !save_out || n_keys < 0) return EAO_EINVAL;
  if (source == TELEMETRY_REPORT && max_age < 0) return EAO_EINVAL;
  if (n_keys > 0 && (!keys || !mask_out)) return EAO_EINVAL;
  if (p->block_tokens < 1 || p->kappa < 0 || p->beta_rank < 0 ||
      p->activity_window < 0 || p->length_window < 1 || p->theta_ppm < 0 ||
      p->mode < EAO_ADMIT_CONDITIONED || p->mode > EAO_ADMIT_FIXED ||
      (p->telemetry != 0 && p->telemetry != 1))
    return EAO_EINVAL;
  if (r->n_tokens < 0 || r->h_tokens < 0 || r->h_tokens > r->n_tokens)
    return EAO_EINVAL;
  if (n_keys != r->n_tokens / p->block_tokens) return EAO_EINVAL;
  if (r->decided < -1 || r->decided > 1) return EAO_EINVAL;
  if (r->decided == -1 && t->have_clock && r->now < t->clock) return EAO_EINVAL;

  /* u: new full chunks the request needs (section 4) */
  int64_t u = r->n_tokens / p->block_tokens - r->h_tokens / p->block_tokens;
  int32_t save;
  if (r->decided >= 0) {
    save = r->decided;  /* the first lookup's choice holds for the request */
  } else {
    if (log_append(t, r->task_id, r->n_tokens, r->now) != EAO_OK) return EAO_ENOMEM;
    t->clock = r->now;
    t->have_clock = 1;

    /* A_t: distinct tasks with a first lookup inside the window */
    int64_t active = 0;
    for (int64_t i = t->log_len - 1; i >= 0; --i) {
      if (!(t->log_time[i] > r->now - p->activity_window)) break;
      int seen = 0;
      for (int64_t j = t->log_len - 1; j > i; --j) {
        if (!(t->log_time[j] > r->now - p->activity_window)) break;
        if (t->log_task[j] == t->log_task[i]) { seen = 1; break; }
      }
      if (!seen) ++active;
    }
    /* N_t: mean prompt length of the last length_window first lookups */
    int64_t cnt = 0;
    int64_t sum = 0;
    for (int64_t i = t->log_len - 1; i >= 0 && cnt < p->length_window; --i) {
      sum += t->log_n[i];
      ++cnt;
    }
    /* [C_reuse > C_H] with C_reuse = (A_t - 1) * (sum / cnt) * beta, exactly:
     * (A_t - 1) * sum * beta > C_H * cnt */
    unsigned __int128 lhs = 0;
    if (active > 1)
      lhs = (unsigned __int128)(active - 1) * (unsigned __int128)sum *
            (unsigned __int128)p->beta_rank;
    unsigned __int128 rhs =
        (unsigned __int128)t->capacity_bytes * (unsigned __int128)cnt;
    int over = lhs > rhs;

    int pressure;
    if (source == TELEMETRY_REPORT) {
      /* the scheduler's copy of the last published report, if fresh */
      int fresh = p->telemetry && rep != NULL && rep->time <= r->now &&
                  r->now - rep->time <= max_age;
      if (fresh) {
        int full = (unsigned __int128)rep->registered * 1000000u >=
                   (unsigned __int128)p->theta_ppm * (unsigned __int128)rep->capacity_slots;
        pressure = over && full && rep->evictions > 0;
      } else {
        pressure = over;  /* no fresh report: the estimate alone decides */
      }
    } else if (p->telemetry) {
      /* tier full and evicting: o_t >= theta and e_t > 0 (Eq. 10) */
      int full = (unsigned __int128)t->registered * 1000000u >=
                 (unsigned __int128)p->theta_ppm * (unsigned __int128)t->K;
      int evicting = t->evictions_total > 0 &&
                     t->evict_stamp[t->evictions_total - 1] > r->now - p->activity_window;
      pressure = over && full && evicting;
    } else {
      pressure = over;  /* no fresh report: the estimate alone decides */
    }
    if (p->mode == EAO_ADMIT_ALWAYS) pressure = 0;
    if (p->mode == EAO_ADMIT_FIXED) pressure = 1;

    save = !(pressure && u > p->kappa);  /* Eq. 6 */

    t->last_window = p->activity_window;
    t->last_active = active;
    t->last_mean = cnt ? (double)sum / (double)cnt : 0.0;
    t->last_ws = (double)(active - 1) * t->last_mean * (double)p->beta_rank;
    t->last_pressure = pressure;
    t->last_save = save;
  }
  /* deduplication: a chunk the tier already holds is not copied again */
  for (int64_t i = 0; i < n_keys; ++i)
    mask_out[i] = (uint8_t)(save && map_find(t, keys + 32 * i) < 0);
  *save_out = save;
  return EAO_OK;
}

int eao_admission_fill(eao_tier *t, const eao_policy *p, const eao_request *r,
                       const uint8_t *keys, int64_t n_keys, uint8_t *mask_out,
                       int32_t *save_out) {
  return admission(t, p, r, TELEMETRY_POLICY, NULL, 0, keys, n_keys, mask_out, save_out);
}

int eao_admission_fill_report(eao_tier *t, const eao_policy *p, const eao_request *r,
                              const eao_tier_report *report, int64_t max_age,
                              const uint8_t *keys, int64_t n_keys, uint8_t *mask_out,
                              int32_t *save_out) {
  return admission(t, p, r, TELEMETRY_REPORT, report, max_age, keys, n_keys, mask_out,
                   save_out);
}

int eao_tier_publish(eao_tier *t, int64_t now, int64_t window, eao_tier_report *out) {
  if (!t || !out || window < 0) return EAO_EINVAL;
  if (t->have_clock && now < t->clock) return EAO_EINVAL;
  t->clock = now;  /* later evictions are stamped no earlier than this */
  t->have_clock = 1;
  int64_t e = 0;
  for (int64_t i = t->evictions_total - 1; i >= 0; --i) {
    if (!(t->evict_stamp[i] > now - window)) break;
    ++e;
  }
  out->time = now;
  out->registered = t->registered;
  out->capacity_slots = t->K;
  out->evictions = e;
  return EAO_OK;
}

/* ------------------------------------------------------------ allocation */

static int record_eviction(eao_tier *t) {
  if (t->evictions_total == t->evict_cap) {
    int64_t cap = t->evict_cap ? 2 * t->evict_cap : 1024;
    int64_t *a = (int64_t *)realloc(t->evict_stamp, (size_t)cap * sizeof(int64_t));
    if (!a) return EAO_ENOMEM;
    t->evict_stamp = a;
    t->evict_cap = cap;
  }
  t->evict_stamp[t->evictions_total] = t->clock;
  t->evictions_total += 1;
  return EAO_OK;
}

int eao_tier_alloc(eao_tier *t, const uint8_t *keys, const uint8_t *mask,
                   int64_t n, int64_t *slots_out, int64_t *allocated) {
  if (!t || n < 0 || !allocated) return EAO_EINVAL;
  if (n > 0 && (!keys || !slots_out)) return EAO_EINVAL;
  int64_t count = 0;
  int exhausted = 0;
  for (int64_t i = 0; i < n; ++i) {
    slots_out[i] = -1;
    if (mask && !mask[i]) continue;
    if (exhausted) continue;
    if (map_find(t, keys + 32 * i) >= 0) continue;  /* held: pending or resident */
    /* lowest-numbered free slot */
    int64_t s = -1;
    for (int64_t c = 0; c < t->K; ++c)
      if (t->state[c] == EAO_SLOT_FREE) { s = c; break; }
    if (s < 0) {
      /* evict the least-recent resident chunk that nothing pins */
      int64_t v = t->head;
      while (v >= 0 && !(t->state[v] == EAO_SLOT_RESIDENT && t->pins[v] == 0))
        v = t->next[v];
      if (v < 0) { exhausted = 1; continue; }
      if (record_eviction(t) != EAO_OK) return EAO_ENOMEM;
      map_remove(t, v);
      lru_unlink(t, v);
      t->state[v] = EAO_SLOT_FREE;
      memset(t->keys + 32 * v, 0, 32);
      t->allocated -= 1;
      t->registered -= 1;
      s = v;
    }
    memcpy(t->keys + 32 * s, keys + 32 * i, 32);
    t->state[s] = EAO_SLOT_PENDING;
    t->pins[s] += 1;
    map_insert(t, s);
    lru_push_recent(t, s);
    t->allocated += 1;  /* not registered until its store is issued */
    slots_out[i] = s;
    ++count;
  }
  *allocated = count;
  return EAO_OK;
}

int eao_tier_mark_stored(eao_tier *t, const int64_t *slots,
                         const uint8_t *mask, int64_t n) {
  if (!t || n < 0) return EAO_EINVAL;
  if (n > 0 && !slots) return EAO_EINVAL;
  for (int64_t i = 0; i < n; ++i) {
    if (mask && !mask[i]) continue;
    if (slots[i] < 0 || slots[i] >= t->K) return EAO_EINVAL;
  }
  for (int64_t i = 0; i < n; ++i) {
    if (mask && !mask[i]) continue;
    if (t->state[slots[i]] == EAO_SLOT_PENDING) {
      t->state[slots[i]] = EAO_SLOT_RESIDENT;
      t->registered += 1;
    }
  }
  return EAO_OK;
}

int eao_tier_unpin(eao_tier *t, const int64_t *slots, int64_t n) {
  if (!t || n < 0) return EAO_EINVAL;
  if (n == 0) return EAO_OK;
  if (!slots) return EAO_EINVAL;
  /* validate on a copy of the pin counts so that nothing changes on error */
  int32_t *left = (int32_t *)malloc((size_t)t->K * sizeof(int32_t));
  if (!left) return EAO_ENOMEM;
  memcpy(left, t->pins, (size_t)t->K * sizeof(int32_t));
  for (int64_t i = 0; i < n; ++i) {
    if (slots[i] < 0 || slots[i] >= t->K || left[slots[i]] <= 0) {
      free(left);
      return EAO_EINVAL;
    }
    left[slots[i]] -= 1;
  }
  free(left);
  for (int64_t i = 0; i < n; ++i) {
    int64_t s = slots[i];
    t->pins[s] -= 1;
    if (t->pins[s] == 0 && t->state[s] == EAO_SLOT_PENDING) {
      /* allocated but never stored: abandon the allocation */
      map_remove(t, s);
      lru_unlink(t, s);
      t->state[s] = EAO_SLOT_FREE;
      memset(t->keys + 32 * s, 0, 32);
      t->allocated -= 1;
    }
  }
  return EAO_OK;
}

int eao_tier_stats_get(const eao_tier *t, eao_tier_stats *s) {
  if (!t || !s) return EAO_EINVAL;
  memset(s, 0, sizeof *s);
  s->capacity_slots = t->K;
  s->allocated = t->allocated;
  s->registered = t->registered;
  for (int64_t i = 0; i < t->K; ++i) s->pinned += t->pins[i] > 0;
  s->evictions_total = t->evictions_total;
  for (int64_t i = t->evictions_total - 1; i >= 0; --i) {
    if (!(t->evict_stamp[i] > t->clock - t->last_window)) break;
    s->evictions_window += 1;
  }
  s->clock = t->clock;
  s->active_tasks = t->last_active;
  s->mean_prompt = t->last_mean;
  s->working_set = t->last_ws;
  s->last_pressure = t->last_pressure;
  s->last_save = t->last_save;
  return EAO_OK;
}

int eao_tier_export(const eao_tier *t, uint8_t *state_out, int32_t *pins_out,
                    uint8_t *keys_out, int64_t *lru_out, int64_t *n_lru) {
  if (!t || !state_out || !pins_out || !keys_out || !lru_out || !n_lru)
    return EAO_EINVAL;
  memcpy(state_out, t->state, (size_t)t->K);
  memcpy(pins_out, t->pins, (size_t)t->K * sizeof(int32_t));
  memcpy(keys_out, t->keys, (size_t)t->K * 32);
  int64_t m = 0;
  for (int64_t s = t->head; s >= 0; s = t->next[s]) lru_out[m++] = s;
  *n_lru = m;
  return EAO_OK;
}
