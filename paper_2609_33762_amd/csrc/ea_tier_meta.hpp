// Host-tier metadata: key -> slot map, LRU recency, pins, free slots, and
// the working-set-aware write admission rule.  Pure CPU code; the caller
// holds the tier lock.
#pragma once

#include <stdint.h>

#include <chrono>
#include <cstring>
#include <deque>
#include <functional>
#include <queue>
#include <unordered_map>
#include <vector>

#include "ea.h"

namespace ea {

// Microseconds on the steady clock: the time base of a wall-clock controller.
inline int64_t steady_now_us() {
  return std::chrono::duration_cast<std::chrono::microseconds>(
             std::chrono::steady_clock::now().time_since_epoch())
      .count();
}

struct Key {
  uint64_t w[4];
  bool operator==(const Key &o) const {
    return w[0] == o.w[0] && w[1] == o.w[1] && w[2] == o.w[2] && w[3] == o.w[3];
  }
  static Key from(const uint8_t *p) {
    Key k;
    std::memcpy(k.w, p, 32);
    return k;
  }
};

struct KeyHash {
  // keys are SHA-256 digests: their first 8 bytes are already uniform
  size_t operator()(const Key &k) const { return (size_t)k.w[0]; }
};

class TierMeta {
 public:
  TierMeta(int64_t slots, int64_t capacity_bytes);

  int64_t capacity() const { return K_; }

  int lookup(const uint8_t *keys, int64_t n, int64_t *hit, int64_t *slots_out);
  // The write rule; with use_report the "full and evicting" factor comes
  // from `rep` when it is fresh (0 <= r.now - rep->time <= max_age), else
  // the working-set estimate alone decides.
  int admission(const ea_policy &p, const ea_request &r, const uint8_t *keys,
                int64_t n_keys, uint8_t *mask_out, int32_t *save_out,
                bool use_report = false, const ea_tier_report *rep = nullptr,
                int64_t max_age = 0);
  // Telemetry at time now (not below the clock); advances the clock.
  int publish(int64_t now, int64_t window, ea_tier_report *out);
  // Stamp evictions with the steady clock in microseconds (a tier driven by
  // a wall-clock controller) instead of the last time the tier was told.
  void use_steady_clock(bool on) { steady_ = on; }
  int alloc(const uint8_t *keys, const uint8_t *mask, int64_t n,
            int64_t *slots_out, int64_t *allocated);
  // A store was issued to `slot`: an allocated slot becomes resident.
  void mark_stored(int64_t slot);
  int unpin(const int64_t *slots, int64_t n);
  void stats(ea_tier_stats_t *s) const;
  void export_state(uint8_t *state, int32_t *pins, uint8_t *keys, int64_t *lru,
                    int64_t *n_lru) const;
  // True when slots [first, first + count) hold nothing (no allocation, no
  // stored chunk).
  bool slots_free(int64_t first, int64_t count) const {
    for (int64_t s = first; s < first + count && s < K_; ++s)
      if (state_[s] != EA_SLOT_FREE) return false;
    return true;
  }

 private:
  // the tier holds a slot under k: pending or resident (deduplication)
  bool held(const Key &k) const { return map_.find(k) != map_.end(); }
  int64_t take_free_slot();
  void release_slot(int64_t s);
  void lru_remove(int64_t s);
  void lru_append(int64_t s);

  int64_t K_;
  int64_t capacity_bytes_;
  std::vector<uint8_t> state_;
  std::vector<int32_t> pins_;
  std::vector<Key> keys_;
  std::vector<int64_t> prev_, next_;
  int64_t lru_head_ = -1, lru_tail_ = -1;  // head = least recent
  std::unordered_map<Key, int64_t, KeyHash> map_;
  // free slots: every slot >= fresh_ was never used; returned_ holds freed
  // slots below fresh_, so the lowest free slot is returned_.top() or fresh_
  int64_t fresh_ = 0;
  std::priority_queue<int64_t, std::vector<int64_t>, std::greater<int64_t>> returned_;
  // Bound the lookup log and the eviction stamps: once either holds more
  // than 65,536 entries, drop those no window used so far can reach again.
  // The clock only moves forward, so an entry at or before
  // clock - keep_time_ is outside every such time window, and only the last
  // keep_count_ lookups enter a mean.
  void trim();

  // allocated_: slots holding a key (pending + resident); registered_:
  // chunks whose store has been issued, the numerator of the occupancy o_t
  // (a store allocates its chunk buffers before it registers the chunks)
  int64_t allocated_ = 0, registered_ = 0;
  std::deque<int64_t> evict_stamps_;
  int64_t evictions_total_ = 0;
  // First lookups in time order; cum is the prompt tokens of every first
  // lookup up to and including this one, so a mean over the last L is one
  // subtraction.
  struct Lookup {
    int64_t time, task, n, cum;
  };
  std::deque<Lookup> log_;
  int64_t log_base_ = 0;  // lookups dropped from the front so far
  int64_t log_cum_ = 0;
  // The tasks of the activity window, kept incrementally for one window
  // length (win_len_, -1 before the first decision): the lookups from index
  // win_first_ (counting dropped ones) to the newest, counted per task.  A
  // decision adds its own lookup and drops those that left the window, so A_t
  // costs amortized constant time per request; a new window length rebuilds
  // the counts once.
  int64_t win_len_ = -1;
  int64_t win_first_ = 0;
  std::unordered_map<int64_t, int64_t> win_tasks_;
  int64_t active_tasks(int64_t window, int64_t horizon);
  int64_t keep_time_ = 0;   // largest activity or report window used
  int64_t keep_count_ = 1;  // largest length window used
  int64_t clock_ = 0;
  bool have_clock_ = false;
  bool steady_ = false;
  int64_t last_window_ = 0, last_active_ = 0;
  double last_mean_ = 0.0, last_ws_ = 0.0;
  int32_t last_pressure_ = 0, last_save_ = 0;
};

}  // namespace ea
