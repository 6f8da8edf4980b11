// Wall-clock write-admission controller (App. "Runtime Admission Details";
// Table "Write-admission parameters").
//
// The worker side publishes the tier's report every report_interval; the
// scheduler side refreshes its copy every read_interval with the latest
// report published at or before that read, and decides each request with
// the copy when it is fresh.  Ticks fall at k * interval after creation.
//
// Manual clock: ea_controller_advance walks the publishes and reads due in
// time order (a publish before a read at the same time), so a run is a pure
// function of its calls.  Steady clock: a thread publishes at its ticks and
// the reads due are resolved when a decision or a status query comes, from
// the last few reports kept for that purpose; the tier reads the steady clock
// itself for decisions, reports and eviction stamps.
#include <algorithm>
#include <condition_variable>
#include <deque>
#include <mutex>
#include <new>
#include <thread>

#include "ea.h"
#include "ea_internal.hpp"
#include "ea_tier_meta.hpp"

namespace {
constexpr size_t kKeep = 64;  // reports kept to answer the reads due
}

struct ea_controller {
  ea_tier *tier = nullptr;
  ea_policy policy{};
  ea_controller_config cfg{};
  int64_t t0 = 0;    // creation time
  int64_t now = 0;   // controller clock (manual) / last time looked at
  int64_t next_publish = 0, next_read = 0;
  std::deque<ea_tier_report> history;  // published reports, oldest first
  int64_t published = 0;
  ea_tier_report seen{};
  bool have_seen = false;
  int64_t decisions = 0, skips = 0, fresh_decisions = 0;
  std::mutex mu;
  std::condition_variable cv;
  bool stop = false;
  std::thread publisher;
};

namespace {

int publish_at(ea_controller *c, int64_t t) {
  ea_tier_report r;
  const int rc = ea_tier_publish(c->tier, t, c->cfg.window, &r);
  if (rc != EA_OK) return rc;
  c->history.push_back(r);
  if (c->history.size() > kKeep) c->history.pop_front();
  c->published += 1;
  return EA_OK;
}

// The scheduler's read at time t: the latest report published at or before t.
void read_at(ea_controller *c, int64_t t) {
  for (auto it = c->history.rbegin(); it != c->history.rend(); ++it) {
    if (it->time <= t) {
      c->seen = *it;
      c->have_seen = true;
      return;
    }
  }
}

// Resolve the reads due up to `t` (the publishes are already done).
void reads_due(ea_controller *c, int64_t t) {
  if (t < c->next_read) return;
  const int64_t ri = c->cfg.read_interval;
  const int64_t last = c->next_read + (t - c->next_read) / ri * ri;
  read_at(c, last);
  c->next_read = last + ri;
}

bool fresh_at(const ea_controller *c, int64_t t) {
  return c->have_seen && c->seen.time <= t && t - c->seen.time <= c->cfg.max_report_age;
}

void publisher_loop(ea_controller *c) {
  std::unique_lock<std::mutex> lk(c->mu);
  while (!c->stop) {
    const int64_t wait_us = c->next_publish - ea::steady_now_us();
    if (wait_us > 0) {
      c->cv.wait_for(lk, std::chrono::microseconds(wait_us));
      continue;  // re-check the stop flag and the time
    }
    // the tier stamps the report with its own steady reading
    if (publish_at(c, c->next_publish) != EA_OK) break;
    c->next_publish += c->cfg.report_interval;
    // after a stall, skip the ticks that have already passed
    const int64_t t = ea::steady_now_us();
    if (c->next_publish <= t)
      c->next_publish += (t - c->next_publish) / c->cfg.report_interval * c->cfg.report_interval +
                         c->cfg.report_interval;
  }
}

}  // namespace

extern "C" {

int ea_controller_create(ea_tier *tier, const ea_policy *policy,
                         const ea_controller_config *cfg, ea_controller **out) {
  if (!tier || !policy || !cfg || !out) return EA_EINVAL;
  if (cfg->report_interval <= 0 || cfg->read_interval <= 0 || cfg->max_report_age < 0 ||
      cfg->window < 0 || (cfg->manual_clock != 0 && cfg->manual_clock != 1))
    return EA_EINVAL;
  ea_controller *c = new (std::nothrow) ea_controller;
  if (!c) return EA_ENOMEM;
  c->tier = tier;
  c->policy = *policy;
  c->policy.activity_window = cfg->window;
  c->cfg = *cfg;
  if (cfg->manual_clock) {
    c->t0 = 0;
  } else {
    ea::tier_use_steady_clock(tier, true);
    c->t0 = ea::steady_now_us();
  }
  c->now = c->t0;
  c->next_publish = c->t0 + cfg->report_interval;
  c->next_read = c->t0 + cfg->read_interval;
  if (!cfg->manual_clock) {
    try {
      c->publisher = std::thread(publisher_loop, c);
    } catch (...) {
      ea::tier_use_steady_clock(tier, false);
      delete c;
      return EA_ENOMEM;
    }
  }
  ea::tier_attach_controller(tier, +1);
  *out = c;
  return EA_OK;
}

int ea_controller_destroy(ea_controller *c) {
  if (!c) return EA_EINVAL;
  {
    std::lock_guard<std::mutex> lk(c->mu);
    c->stop = true;
  }
  c->cv.notify_all();
  if (c->publisher.joinable()) c->publisher.join();
  if (!c->cfg.manual_clock) ea::tier_use_steady_clock(c->tier, false);
  ea::tier_attach_controller(c->tier, -1);
  delete c;
  return EA_OK;
}

int ea_controller_advance(ea_controller *c, int64_t now) {
  try {
    if (!c || !c->cfg.manual_clock) return EA_EINVAL;
    std::lock_guard<std::mutex> lk(c->mu);
    if (now < c->now) return EA_EINVAL;
    while (true) {
      const int64_t t = std::min(c->next_publish, c->next_read);
      if (t > now) break;
      if (c->next_publish <= c->next_read) {  // a publish first at equal times
        const int rc = publish_at(c, c->next_publish);
        if (rc != EA_OK) return rc;
        c->next_publish += c->cfg.report_interval;
      } else {
        read_at(c, c->next_read);
        c->next_read += c->cfg.read_interval;
      }
    }
    c->now = now;
    return EA_OK;
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
}

int ea_controller_decide(ea_controller *c, int64_t n_tokens, int64_t h_tokens,
                         int64_t task_id, int32_t decided, const uint8_t *keys,
                         int64_t n_keys, uint8_t *mask_out, int32_t *save_out) {
  try {
    if (!c || !save_out) return EA_EINVAL;
    std::lock_guard<std::mutex> lk(c->mu);
    if (!c->cfg.manual_clock) {
      c->now = std::max(c->now, ea::steady_now_us());
      reads_due(c, c->now);
    }
    ea_request r{n_tokens, h_tokens, task_id, c->now, decided, 0};
    const int rc = ea_admission_fill_report(c->tier, &c->policy, &r,
                                            c->have_seen ? &c->seen : nullptr,
                                            c->cfg.max_report_age, keys, n_keys, mask_out,
                                            save_out);
    if (rc == EA_OK && decided == -1) {
      c->decisions += 1;
      c->skips += *save_out ? 0 : 1;
      c->fresh_decisions += (c->policy.telemetry && fresh_at(c, c->now)) ? 1 : 0;
    }
    return rc;
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
}

int ea_controller_get_status(ea_controller *c, ea_controller_status *s) {
  if (!c || !s) return EA_EINVAL;
  std::lock_guard<std::mutex> lk(c->mu);
  if (!c->cfg.manual_clock) {
    c->now = std::max(c->now, ea::steady_now_us());
    reads_due(c, c->now);
  }
  *s = ea_controller_status{};
  s->now = c->now;
  s->reports_published = c->published;
  if (!c->history.empty()) s->published = c->history.back();
  s->seen = c->seen;
  s->have_seen = c->have_seen ? 1 : 0;
  s->fresh = fresh_at(c, c->now) ? 1 : 0;
  s->decisions = c->decisions;
  s->skips = c->skips;
  s->fresh_decisions = c->fresh_decisions;
  return EA_OK;
}

}  // extern "C"
