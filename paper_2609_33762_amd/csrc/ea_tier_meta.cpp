// Host-tier metadata and write admission (see ea_tier_meta.hpp).
//
// The LRU host tier of App. "Runtime Admission Details" and "Recency order
// of the host tier": a recency list with new chunks appended at the tail; a
// lookup promotes only its leading hits to the tail; chunks leave only when an
// allocation finds no free slot, which then takes the first resident chunk
// from the head that no lookup, allocation or transfer pins.
#include "ea_tier_meta.hpp"

#include <algorithm>

namespace ea {

TierMeta::TierMeta(int64_t slots, int64_t capacity_bytes)
    : K_(slots),
      capacity_bytes_(capacity_bytes),
      state_(slots, EA_SLOT_FREE),
      pins_(slots, 0),
      keys_(slots, Key{{0, 0, 0, 0}}),
      prev_(slots, -1),
      next_(slots, -1) {
  map_.reserve((size_t)slots * 2);
}

void TierMeta::lru_remove(int64_t s) {
  const int64_t p = prev_[s], n = next_[s];
  if (p >= 0) next_[p] = n; else lru_head_ = n;
  if (n >= 0) prev_[n] = p; else lru_tail_ = p;
  prev_[s] = next_[s] = -1;
}

void TierMeta::lru_append(int64_t s) {
  prev_[s] = lru_tail_;
  next_[s] = -1;
  if (lru_tail_ >= 0) next_[lru_tail_] = s; else lru_head_ = s;
  lru_tail_ = s;
}

int64_t TierMeta::take_free_slot() {
  if (!returned_.empty()) {
    const int64_t s = returned_.top();
    returned_.pop();
    return s;
  }
  if (fresh_ < K_) return fresh_++;
  return -1;
}

void TierMeta::trim() {
  constexpr size_t kTrimAt = size_t(1) << 16;  // history kept whole up to this size
  if (!have_clock_) return;
  const __int128 old = (__int128)clock_ - keep_time_;
  if (log_.size() > kTrimAt)
    while ((int64_t)log_.size() > keep_count_ && (__int128)log_.front().time <= old) {
      if (win_len_ >= 0 && log_base_ >= win_first_) {
        // still counted in the activity window: it would leave at the next
        // decision anyway, since its time is at or before clock - keep_time_
        auto it = win_tasks_.find(log_.front().task);
        if (--it->second == 0) win_tasks_.erase(it);
        win_first_ = log_base_ + 1;
      }
      log_.pop_front();
      ++log_base_;
    }
  if (evict_stamps_.size() > kTrimAt)
    while (!evict_stamps_.empty() && (__int128)evict_stamps_.front() <= old)
      evict_stamps_.pop_front();
}

void TierMeta::release_slot(int64_t s) {
  map_.erase(keys_[s]);
  lru_remove(s);
  state_[s] = EA_SLOT_FREE;
  keys_[s] = Key{{0, 0, 0, 0}};
  allocated_ -= 1;  // only pending slots are released here
  returned_.push(s);
}

int TierMeta::lookup(const uint8_t *keys, int64_t n, int64_t *hit,
                     int64_t *slots_out) {
  int64_t h = 0;
  for (; h < n; ++h) {
    auto it = map_.find(Key::from(keys + 32 * h));
    if (it == map_.end() || state_[it->second] != EA_SLOT_RESIDENT) break;
    slots_out[h] = it->second;
  }
  for (int64_t i = 0; i < h; ++i) {
    const int64_t s = slots_out[i];
    lru_remove(s);
    lru_append(s);
    pins_[s] += 1;
  }
  *hit = h;
  return EA_OK;
}

int TierMeta::admission(const ea_policy &p, const ea_request &r,
                        const uint8_t *keys, int64_t n_keys, uint8_t *mask_out,
                        int32_t *save_out, bool use_report, const ea_tier_report *rep,
                        int64_t max_age) {
  if (use_report && max_age < 0) return EA_EINVAL;
  if (p.block_tokens < 1 || p.kappa < 0 || p.beta_rank < 0 ||
      p.activity_window < 0 || p.length_window < 1 || p.theta_ppm < 0 ||
      p.mode < EA_ADMIT_CONDITIONED || p.mode > EA_ADMIT_FIXED ||
      (p.telemetry != 0 && p.telemetry != 1))
    return EA_EINVAL;
  if (r.n_tokens < 0 || r.h_tokens < 0 || r.h_tokens > r.n_tokens) return EA_EINVAL;
  if (n_keys != r.n_tokens / p.block_tokens) return EA_EINVAL;
  if (r.decided < -1 || r.decided > 1) return EA_EINVAL;
  // on the steady clock the tier reads the time itself, under its lock, so
  // decisions, reports and evictions stay in order whatever the threads do
  const int64_t now =
      steady_ ? std::max(have_clock_ ? clock_ : INT64_MIN, steady_now_us()) : r.now;
  if (r.decided == -1 && have_clock_ && now < clock_) return EA_EINVAL;

  // new full chunks the request needs (section 4)
  const int64_t u = r.n_tokens / p.block_tokens - r.h_tokens / p.block_tokens;
  int32_t save;
  if (r.decided >= 0) {
    save = r.decided;  // a later lookup of the request keeps the first choice
  } else {
    log_cum_ += r.n_tokens;
    log_.push_back(Lookup{now, r.task_id, r.n_tokens, log_cum_});
    clock_ = now;
    have_clock_ = true;
    keep_time_ = std::max(keep_time_, p.activity_window);
    keep_count_ = std::max<int64_t>(keep_count_, p.length_window);
    const int64_t horizon = now - p.activity_window;

    // A_t: distinct tasks whose first lookup falls inside the window
    const int64_t active = active_tasks(p.activity_window, horizon);

    // N_t: mean prompt length of the last length_window first lookups
    const int64_t size = (int64_t)log_.size();
    const int64_t cnt = std::min<int64_t>(p.length_window, size);
    const int64_t before = cnt < size ? log_[(size_t)(size - 1 - cnt)].cum
                                      : log_.front().cum - log_.front().n;
    const int64_t sum = log_.back().cum - before;

    // [C_reuse > C_H], C_reuse = (A_t - 1) * (sum / cnt) * beta (Eq. 5),
    // compared exactly as (A_t - 1) * sum * beta > C_H * cnt
    using u128 = unsigned __int128;
    const u128 lhs = active > 1 ? (u128)(active - 1) * (u128)sum * (u128)p.beta_rank : 0;
    const u128 rhs = (u128)capacity_bytes_ * (u128)cnt;
    const bool over = lhs > rhs;

    bool pressure;
    if (use_report) {
      // the scheduler's copy of the worker's last report, when fresh
      const bool fresh = p.telemetry && rep != nullptr && rep->time <= now &&
                         now - rep->time <= max_age;
      if (fresh) {
        const bool full = (u128)rep->registered * 1000000u >=
                          (u128)p.theta_ppm * (u128)rep->capacity_slots;
        pressure = over && full && rep->evictions > 0;
      } else {
        pressure = over;
      }
    } else if (p.telemetry) {
      // tier full and evicting: o_t >= theta and e_t > 0 (Eq. 10)
      const bool full = (u128)registered_ * 1000000u >= (u128)p.theta_ppm * (u128)K_;
      const bool evicting = !evict_stamps_.empty() && evict_stamps_.back() > horizon;
      pressure = over && full && evicting;
    } else {
      pressure = over;  // no fresh report: the estimate alone decides
    }
    if (p.mode == EA_ADMIT_ALWAYS) pressure = false;
    if (p.mode == EA_ADMIT_FIXED) pressure = true;

    save = !(pressure && u > p.kappa);  // Eq. 6

    last_window_ = p.activity_window;
    last_active_ = active;
    last_mean_ = cnt ? (double)sum / (double)cnt : 0.0;
    last_ws_ = (double)(active - 1) * last_mean_ * (double)p.beta_rank;
    last_pressure_ = pressure ? 1 : 0;
    last_save_ = save;
    trim();
  }
  // copy-time deduplication: chunks the tier already holds are not copied
  for (int64_t i = 0; i < n_keys; ++i)
    mask_out[i] = (uint8_t)(save && !held(Key::from(keys + 32 * i)));
  *save_out = save;
  return EA_OK;
}

int64_t TierMeta::active_tasks(int64_t window, int64_t horizon) {
  const int64_t end = log_base_ + (int64_t)log_.size();  // one past the newest
  auto at = [&](int64_t i) -> const Lookup & { return log_[(size_t)(i - log_base_)]; };
  if (window != win_len_) {
    // a window length not seen last time: count it from scratch
    win_tasks_.clear();
    int64_t i = end;
    while (i > log_base_ && at(i - 1).time > horizon) {
      --i;
      win_tasks_[at(i).task] += 1;
    }
    win_first_ = i;
    win_len_ = window;
  } else {
    win_tasks_[at(end - 1).task] += 1;  // this decision's own lookup
    while (win_first_ < end && at(win_first_).time <= horizon) {
      auto it = win_tasks_.find(at(win_first_).task);
      if (--it->second == 0) win_tasks_.erase(it);
      ++win_first_;
    }
  }
  return (int64_t)win_tasks_.size();
}

int TierMeta::publish(int64_t now, int64_t window, ea_tier_report *out) {
  if (window < 0) return EA_EINVAL;
  if (steady_) now = std::max(have_clock_ ? clock_ : INT64_MIN, steady_now_us());
  if (have_clock_ && now < clock_) return EA_EINVAL;
  clock_ = now;
  have_clock_ = true;
  keep_time_ = std::max(keep_time_, window);
  int64_t e = 0;
  for (auto it = evict_stamps_.rbegin(); it != evict_stamps_.rend() && *it > now - window; ++it)
    ++e;
  out->time = now;
  out->registered = registered_;
  out->capacity_slots = K_;
  out->evictions = e;
  trim();
  return EA_OK;
}

int TierMeta::alloc(const uint8_t *keys, const uint8_t *mask, int64_t n,
                    int64_t *slots_out, int64_t *allocated) {
  if (steady_) {
    clock_ = std::max(clock_, steady_now_us());
    have_clock_ = true;
  }
  int64_t count = 0;
  bool exhausted = false;
  for (int64_t i = 0; i < n; ++i) {
    slots_out[i] = -1;
    if ((mask && !mask[i]) || exhausted) continue;
    const Key k = Key::from(keys + 32 * i);
    if (held(k)) continue;
    int64_t s = take_free_slot();
    if (s < 0) {
      // evict the least-recent resident chunk nothing pins
      int64_t v = lru_head_;
      while (v >= 0 && !(state_[v] == EA_SLOT_RESIDENT && pins_[v] == 0)) v = next_[v];
      if (v < 0) {
        exhausted = true;
        continue;
      }
      evict_stamps_.push_back(clock_);
      evictions_total_ += 1;
      map_.erase(keys_[v]);
      lru_remove(v);
      state_[v] = EA_SLOT_FREE;
      allocated_ -= 1;
      registered_ -= 1;
      s = v;
    }
    keys_[s] = k;
    state_[s] = EA_SLOT_PENDING;
    pins_[s] += 1;
    map_.emplace(k, s);
    lru_append(s);
    allocated_ += 1;  // registered once its store is issued (mark_stored)
    slots_out[i] = s;
    ++count;
  }
  *allocated = count;
  trim();
  return EA_OK;
}

void TierMeta::mark_stored(int64_t slot) {
  if (state_[slot] == EA_SLOT_PENDING) {
    state_[slot] = EA_SLOT_RESIDENT;
    registered_ += 1;
  }
}

int TierMeta::unpin(const int64_t *slots, int64_t n) {
  std::unordered_map<int64_t, int32_t> drop;
  for (int64_t i = 0; i < n; ++i) {
    const int64_t s = slots[i];
    if (s < 0 || s >= K_) return EA_EINVAL;
    if (++drop[s] > pins_[s]) return EA_EINVAL;
  }
  for (int64_t i = 0; i < n; ++i) {
    const int64_t s = slots[i];
    pins_[s] -= 1;
    if (pins_[s] == 0 && state_[s] == EA_SLOT_PENDING) release_slot(s);  // abandoned
  }
  return EA_OK;
}

void TierMeta::stats(ea_tier_stats_t *s) const {
  s->capacity_slots = K_;
  s->allocated = allocated_;
  s->registered = registered_;
  int64_t pinned = 0;
  for (int32_t p : pins_) pinned += p > 0;
  s->pinned = pinned;
  s->evictions_total = evictions_total_;
  int64_t in_window = 0;
  for (auto it = evict_stamps_.rbegin();
       it != evict_stamps_.rend() && *it > clock_ - last_window_; ++it)
    ++in_window;
  s->evictions_window = in_window;
  s->clock = clock_;
  s->active_tasks = last_active_;
  s->mean_prompt = last_mean_;
  s->working_set = last_ws_;
  s->last_pressure = last_pressure_;
  s->last_save = last_save_;
}

void TierMeta::export_state(uint8_t *state, int32_t *pins, uint8_t *keys,
                            int64_t *lru, int64_t *n_lru) const {
  std::memcpy(state, state_.data(), (size_t)K_);
  std::memcpy(pins, pins_.data(), (size_t)K_ * sizeof(int32_t));
  for (int64_t s = 0; s < K_; ++s) std::memcpy(keys + 32 * s, keys_[s].w, 32);
  int64_t m = 0;
  for (int64_t s = lru_head_; s >= 0; s = next_[s]) lru[m++] = s;
  *n_lru = m;
}

}  // namespace ea
