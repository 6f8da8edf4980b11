// Differential fuzz of the library's host-side code against the oracle,
// meant to be built with AddressSanitizer and UndefinedBehaviorSanitizer.
//
// Test infrastructure only: it links the product's host-only sources
// (ea_tier_meta.cpp: key map, LRU recency, pins, free slots and the write
// admission of section 4, Eq. 6 and Eq. 10; ea_stack.cpp: the reuse-distance
// capacity tool of section 3.2, Eq. 4) together with the oracle, drives both
// with the same seeded random request streams, and stops at the first
// difference.  The oracle's own hashing and copies run on random ragged
// inputs too.  No GPU is involved: the tier metadata needs no device memory.
//
// Usage: tier_fuzz <seed> <requests>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <algorithm>
#include <random>
#include <vector>

#include "ea.h"
#include "ea_tier_meta.hpp"
#include "eao.h"

namespace {

[[noreturn]] void fail(const char *what, int64_t at) {
  std::fprintf(stderr, "MISMATCH: %s at request %lld\n", what, (long long)at);
  std::exit(1);
}
#define CHECK(cond, what, at) \
  do {                        \
    if (!(cond)) fail(what, at); \
  } while (0)

using Rng = std::mt19937_64;

int64_t uniform(Rng &r, int64_t lo, int64_t hi) {  // inclusive
  return std::uniform_int_distribution<int64_t>(lo, hi)(r);
}
bool coin(Rng &r, double p) { return std::uniform_real_distribution<double>(0, 1)(r) < p; }

struct Key32 {
  uint8_t b[32];
};

Key32 fresh_key(Rng &r) {
  Key32 k;
  for (int i = 0; i < 4; ++i) {
    const uint64_t v = r();
    std::memcpy(k.b + 8 * i, &v, 8);
  }
  return k;
}

const uint8_t *raw(const std::vector<Key32> &v) {
  return v.empty() ? nullptr : v[0].b;
}

void compare_state(ea::TierMeta &m, eao_tier *o, int64_t K, int64_t at) {
  std::vector<uint8_t> st1(K), st2(K), k1(32 * K), k2(32 * K);
  std::vector<int32_t> p1(K), p2(K);
  std::vector<int64_t> l1(K), l2(K);
  int64_t n1 = 0, n2 = 0;
  m.export_state(st1.data(), p1.data(), k1.data(), l1.data(), &n1);
  CHECK(eao_tier_export(o, st2.data(), p2.data(), k2.data(), l2.data(), &n2) == 0, "export", at);
  CHECK(st1 == st2, "slot states", at);
  CHECK(p1 == p2, "pins", at);
  CHECK(k1 == k2, "keys", at);
  CHECK(n1 == n2 && std::equal(l1.begin(), l1.begin() + n1, l2.begin()), "LRU order", at);
  ea_tier_stats_t a;
  std::memset(&a, 0, sizeof a);
  m.stats(&a);
  eao_tier_stats b;
  CHECK(eao_tier_stats_get(o, &b) == 0, "stats", at);
  CHECK(a.capacity_slots == b.capacity_slots && a.registered == b.registered &&
            a.allocated == b.allocated && a.pinned == b.pinned &&
            a.evictions_total == b.evictions_total &&
            a.evictions_window == b.evictions_window && a.clock == b.clock &&
            a.active_tasks == b.active_tasks && a.last_pressure == b.last_pressure &&
            a.last_save == b.last_save,
        "statistics", at);
}

// The tier: random agents whose prompts grow, get edited and repeat.
void fuzz_tier(uint64_t seed, int64_t requests) {
  Rng r(seed);
  const int64_t slot_bytes = 2048;  // the oracle shape below: 2*16*1*32*2
  const int64_t K = requests > 20000 ? uniform(r, 4, 12) : uniform(r, 1, 40);
  const int64_t cap = K * slot_bytes + uniform(r, 0, slot_bytes - 1);
  eao_shape sh{64, 1, 16, 1, 32, 2, 0, 1};
  CHECK(eao_slot_bytes(&sh) == slot_bytes, "oracle slot size", -1);
  eao_tier *o = nullptr;
  CHECK(eao_tier_create(&sh, cap, &o) == 0 && eao_tier_capacity(o) == K, "oracle tier", -1);
  ea::TierMeta m(K, cap);

  const int64_t b = 16;
  ea_policy p{};
  const int64_t thetas[3] = {500000, 950000, 1000000};
  p.theta_ppm = thetas[uniform(r, 0, 2)];
  p.kappa = uniform(r, 0, 4);
  p.block_tokens = b;
  p.beta_rank = uniform(r, 1, 4) * 64;
  p.activity_window = uniform(r, 1, 30);
  p.length_window = (int32_t)uniform(r, 1, 40);
  p.mode = (int32_t)uniform(r, 0, 2);
  p.telemetry = (int32_t)uniform(r, 0, 1);
  eao_policy q;
  static_assert(sizeof(q) == sizeof(p), "policy layouts");
  std::memcpy(&q, &p, sizeof p);
  const int64_t report_window = uniform(r, 1, 30);

  const int n_agents = (int)uniform(r, 1, 10);
  std::vector<std::vector<Key32>> prompt(n_agents);
  std::vector<int64_t> held;      // slots still pinned (pins drop later)
  std::vector<int64_t> deferred;  // allocated slots whose store comes later
  int64_t now = 0;
  bool have_rep = false;
  ea_tier_report rep{};
  for (int64_t t = 0; t < requests; ++t) {
    if (requests <= 20000 && coin(r, 0.05)) {
      // a caller may change the windows between requests (the tier then
      // recounts the activity window); the long stream keeps them, since
      // windows larger than any before could reach history the tier dropped
      p.activity_window = uniform(r, 0, 30);
      p.length_window = (int32_t)uniform(r, 1, 40);
      std::memcpy(&q, &p, sizeof p);
    }
    const int a = (int)uniform(r, 0, n_agents - 1);
    auto &pk = prompt[a];
    if (!pk.empty() && coin(r, 0.1)) {  // an edit rekeys the rest of the prompt
      const int64_t at = uniform(r, 0, (int64_t)pk.size() - 1);
      for (int64_t i = at; i < (int64_t)pk.size(); ++i) pk[i] = fresh_key(r);
    }
    const int64_t grow = requests > 20000 ? uniform(r, 0, 1) : uniform(r, 0, 3);
    for (int64_t i = 0; i < grow; ++i) pk.push_back(fresh_key(r));
    if ((int64_t)pk.size() > 12) pk.erase(pk.begin(), pk.begin() + ((int64_t)pk.size() - 12));
    const std::vector<Key32> keys = pk;
    const int64_t n = (int64_t)keys.size();

    // lookup
    std::vector<int64_t> s1(n + 1, -7), s2(n + 1, -7);
    int64_t h1 = -1, h2 = -1;
    CHECK(m.lookup(raw(keys), n, &h1, s1.data()) == 0, "lookup rc", t);
    CHECK(eao_tier_lookup(o, raw(keys), n, &h2, s2.data()) == 0, "oracle lookup rc", t);
    CHECK(h1 == h2 && std::equal(s1.begin(), s1.begin() + h1, s2.begin()), "lookup", t);

    // admission (sometimes with a published report, sometimes invalid)
    now += uniform(r, 0, 3);
    ea_request rq{n * b + uniform(r, 0, b - 1), h1 * b, a, now, -1, 0};
    if (coin(r, 0.03)) rq.h_tokens = rq.n_tokens + 1;  // invalid: h > n
    eao_request oq;
    std::memcpy(&oq, &rq, sizeof rq);
    std::vector<uint8_t> m1(n + 1, 9), m2(n + 1, 9);
    int32_t v1 = -1, v2 = -1;
    const bool use_rep = coin(r, 0.3);
    const int64_t max_age = uniform(r, 0, 20);
    int rc1, rc2;
    if (use_rep) {
      eao_tier_report orep;
      std::memcpy(&orep, &rep, sizeof rep);
      rc1 = m.admission(p, rq, raw(keys), n, m1.data(), &v1, true, have_rep ? &rep : nullptr,
                        max_age);
      rc2 = eao_admission_fill_report(o, &q, &oq, have_rep ? &orep : nullptr, max_age,
                                      raw(keys), n, m2.data(), &v2);
    } else {
      rc1 = m.admission(p, rq, raw(keys), n, m1.data(), &v1);
      rc2 = eao_admission_fill(o, &q, &oq, raw(keys), n, m2.data(), &v2);
    }
    CHECK(rc1 == rc2, "admission rc", t);
    if (rc1 != 0) {  // refused: the lookup's pins stay until a later release
      held.insert(held.end(), s1.begin(), s1.begin() + h1);
      compare_state(m, o, K, t);
      continue;
    }
    CHECK(v1 == v2 && std::equal(m1.begin(), m1.begin() + n, m2.begin()), "admission", t);
    if (coin(r, 0.1)) {  // a later lookup of the same request keeps the choice
      rq.decided = v1;
      oq.decided = v2;
      CHECK(m.admission(p, rq, raw(keys), n, m1.data(), &v1) == 0, "repeat admission rc", t);
      CHECK(eao_admission_fill(o, &q, &oq, raw(keys), n, m2.data(), &v2) == 0,
            "oracle repeat admission rc", t);
      CHECK(v1 == v2 && std::equal(m1.begin(), m1.begin() + n, m2.begin()), "repeat", t);
    }

    // allocation, stores, pins
    int64_t c1 = -1, c2 = -1;
    std::vector<int64_t> a1(n + 1, -7), a2(n + 1, -7);
    CHECK(m.alloc(raw(keys), m1.data(), n, a1.data(), &c1) == 0, "alloc rc", t);
    CHECK(eao_tier_alloc(o, raw(keys), m1.data(), n, a2.data(), &c2) == 0, "oracle alloc rc", t);
    CHECK(c1 == c2 && std::equal(a1.begin(), a1.begin() + n, a2.begin()), "alloc", t);
    std::vector<int64_t> got;
    for (int64_t i = 0; i < n; ++i)
      if (a1[i] >= 0) got.push_back(a1[i]);
    if (coin(r, 0.25)) {
      // the store is issued some requests later: decisions and reports in
      // between see these slots allocated but not registered
      deferred.insert(deferred.end(), got.begin(), got.end());
      got.clear();
    }
    for (int64_t s : got)
      if (coin(r, 0.9)) {
        m.mark_stored(s);
        CHECK(eao_tier_mark_stored(o, &s, nullptr, 1) == 0, "mark stored", t);
      }
    for (int64_t s : got) {
      if (coin(r, 0.95)) {
        CHECK(m.unpin(&s, 1) == 0 && eao_tier_unpin(o, &s, 1) == 0, "unpin", t);
      } else {
        held.push_back(s);
      }
    }
    if (!deferred.empty() && coin(r, 0.3)) {
      for (int64_t s : deferred) {
        m.mark_stored(s);
        CHECK(eao_tier_mark_stored(o, &s, nullptr, 1) == 0, "deferred store", t);
        CHECK(m.unpin(&s, 1) == 0 && eao_tier_unpin(o, &s, 1) == 0, "deferred unpin", t);
      }
      deferred.clear();
    }
    for (int64_t i = 0; i < h1; ++i) {
      if (coin(r, 0.8)) {
        CHECK(m.unpin(&s1[i], 1) == 0 && eao_tier_unpin(o, &s1[i], 1) == 0, "unpin hit", t);
      } else {
        held.push_back(s1[i]);
      }
    }
    if (coin(r, 0.03) && !held.empty()) {
      CHECK(m.unpin(held.data(), (int64_t)held.size()) == 0, "unpin held", t);
      CHECK(eao_tier_unpin(o, held.data(), (int64_t)held.size()) == 0, "oracle unpin held", t);
      held.clear();
    }
    if (coin(r, 0.02)) {  // one pin more than the slot holds: refused, nothing changes
      const int64_t s0 = uniform(r, 0, K - 1);
      std::vector<uint8_t> st(K), kk(32 * K);
      std::vector<int32_t> pins(K);
      std::vector<int64_t> lru(K);
      int64_t nl = 0;
      m.export_state(st.data(), pins.data(), kk.data(), lru.data(), &nl);
      std::vector<int64_t> too((size_t)pins[s0] + 1, s0);
      CHECK(m.unpin(too.data(), (int64_t)too.size()) != 0, "over-unpin accepted", t);
      CHECK(eao_tier_unpin(o, too.data(), (int64_t)too.size()) != 0,
            "oracle over-unpin accepted", t);
    }

    // the worker's report
    if (coin(r, 0.2)) {
      now += uniform(r, 0, 2);
      eao_tier_report orep;
      CHECK(m.publish(now, report_window, &rep) == 0, "publish rc", t);
      CHECK(eao_tier_publish(o, now, report_window, &orep) == 0, "oracle publish rc", t);
      CHECK(rep.time == orep.time && rep.registered == orep.registered &&
                rep.capacity_slots == orep.capacity_slots && rep.evictions == orep.evictions,
            "report", t);
      have_rep = true;
    }
    if (requests <= 20000 || t % 1000 == 0 || t == requests - 1) compare_state(m, o, K, t);
  }
  eao_tier_destroy(o);
}

// The capacity tool against the oracle's reference models and brute force.
void fuzz_stack(uint64_t seed) {
  Rng r(seed ^ 0x5eedull);
  const int64_t n_req = uniform(r, 0, 60);
  const int64_t universe = uniform(r, 1, 40);
  std::vector<Key32> pool(universe);
  for (auto &k : pool) k = fresh_key(r);
  std::vector<int64_t> off(1, 0);
  std::vector<Key32> refs;
  std::vector<uint8_t> declined_req(n_req), declined_ref;
  for (int64_t j = 0; j < n_req; ++j) {
    const int64_t len = uniform(r, 0, 12);
    declined_req[j] = coin(r, 0.3);
    for (int64_t i = 0; i < len; ++i) {
      refs.push_back(pool[uniform(r, 0, universe - 1)]);
      declined_ref.push_back(declined_req[j]);
    }
    off.push_back((int64_t)refs.size());
  }
  const int64_t n = (int64_t)refs.size();
  std::vector<int64_t> prev(n + 1), next(n + 1);
  CHECK(ea_reuse_distances(raw(refs), n, prev.data(), next.data()) == 0, "distances rc", -1);
  for (int64_t i = 0; i < n; ++i) {  // brute force: distinct chunks in between
    int64_t s = i - 1;
    while (s >= 0 && std::memcmp(refs[s].b, refs[i].b, 32) != 0) --s;
    int64_t d = -1;
    if (s >= 0) {
      std::vector<Key32> seen;
      for (int64_t x = s + 1; x < i; ++x) {
        bool dup = false;
        for (auto &y : seen) dup = dup || std::memcmp(y.b, refs[x].b, 32) == 0;
        if (!dup) seen.push_back(refs[x]);
      }
      d = (int64_t)seen.size();
      CHECK(next[s] == d, "next distance", -1);
    }
    CHECK(prev[i] == d, "reuse distance", -1);
  }
  for (int64_t cap = 0; cap <= universe + 1; ++cap) {
    std::vector<uint8_t> h1(n + 1), h2(n + 1);
    const uint8_t *dec = coin(r, 0.5) ? declined_ref.data() : nullptr;
    CHECK(ea_lru_simulate(raw(refs), n, dec, cap, h1.data()) == 0, "simulate rc", cap);
    CHECK(eao_lru_reference(raw(refs), n, dec, cap, h2.data()) == 0, "reference rc", cap);
    CHECK(std::equal(h1.begin(), h1.begin() + n, h2.begin()), "reference model", cap);
    std::vector<int64_t> q1(n_req + 1), q2(n_req + 1);
    const uint8_t *dr = coin(r, 0.5) ? declined_req.data() : nullptr;
    CHECK(ea_lru_simulate_prefix(raw(refs), off.data(), n_req, dr, cap, q1.data()) == 0,
          "prefix model rc", cap);
    CHECK(eao_lru_prefix_model(raw(refs), off.data(), n_req, dr, cap, q2.data()) == 0,
          "oracle prefix model rc", cap);
    CHECK(std::equal(q1.begin(), q1.begin() + n_req, q2.begin()), "prefix model", cap);
    std::vector<int64_t> cov(n_req + 1);
    const int64_t caps[1] = {cap};
    CHECK(ea_prefix_coverage(prev.data(), off.data(), n_req, caps, 1, cov.data()) == 0,
          "coverage rc", cap);
    for (int64_t j = 0; j < n_req; ++j) {
      int64_t c = 0;
      while (off[j] + c < off[j + 1] && prev[off[j] + c] >= 0 && prev[off[j] + c] < cap) ++c;
      CHECK(cov[j] == c, "coverage", cap);
    }
  }
}

// The oracle's hashing and copies on random ragged inputs (memory safety
// under the sanitizers, buffers sized exactly), with two invariants: keys
// appear only for full blocks, and a store followed by a load into other
// pages reproduces the source pages and scales byte for byte.
void fuzz_oracle_bytes(uint64_t seed) {
  Rng r(seed ^ 0xb17e5ull);
  // hashing
  const int32_t n_seqs = (int32_t)uniform(r, 0, 6);
  const int32_t b = (int32_t)uniform(r, 1, 40);
  std::vector<int64_t> off(1, 0);
  for (int32_t q = 0; q < n_seqs; ++q) off.push_back(off.back() + uniform(r, 0, 130));
  std::vector<int32_t> tok((size_t)off.back());
  for (auto &x : tok) x = (int32_t)r();
  int64_t total = 0;
  for (int32_t q = 0; q < n_seqs; ++q) total += (off[q + 1] - off[q]) / b;
  std::vector<uint8_t> parents(32 * (size_t)n_seqs), keys(32 * (size_t)total);
  for (auto &x : parents) x = (uint8_t)r();
  std::vector<int64_t> koff((size_t)n_seqs + 1);
  CHECK(eao_hash_blocks(tok.empty() ? nullptr : tok.data(), off.data(), n_seqs, b,
                        coin(r, 0.5) && n_seqs ? parents.data() : nullptr,
                        keys.empty() ? nullptr : keys.data(), koff.data()) == 0,
        "hash rc", -1);
  for (int32_t q = 0; q < n_seqs; ++q)
    CHECK(koff[q + 1] - koff[q] == (off[q + 1] - off[q]) / b, "key offsets", -1);

  // store then load
  eao_shape sh;
  sh.num_pages = (int32_t)uniform(r, 4, 40);
  sh.num_layers = (int32_t)uniform(r, 1, 3);
  const int32_t ts[4] = {1, 2, 4, 16};
  sh.page_tokens = ts[uniform(r, 0, 3)];
  sh.num_kv_heads = (int32_t)uniform(r, 1, 2);
  sh.head_dim = coin(r, 0.5) ? 8 : 16;
  sh.elem_bytes = coin(r, 0.5) ? 1 : 2;
  sh.has_scales = coin(r, 0.5) ? 1 : 0;
  sh.chunk_pages = (int32_t)uniform(r, 1, 3);
  const int64_t C = sh.chunk_pages, L = sh.num_layers, P = sh.num_pages;
  const int64_t piece = eao_piece_bytes(&sh);
  const int64_t S = uniform(r, 1, 6);
  std::vector<uint8_t> cache((size_t)eao_cache_bytes(&sh)), tier((size_t)(S * eao_slot_bytes(&sh)));
  std::vector<uint8_t> scales((size_t)eao_scale_bytes(&sh));
  for (auto &x : cache) x = (uint8_t)r();
  for (auto &x : scales) x = (uint8_t)r();
  const int64_t n = std::min<int64_t>(S, P / (2 * C));
  if (n < 1) return;
  std::vector<int64_t> slots(S);
  for (int64_t i = 0; i < S; ++i) slots[i] = i;
  std::shuffle(slots.begin(), slots.end(), r);
  slots.resize(n);
  std::vector<int32_t> pages(P);
  for (int64_t i = 0; i < P; ++i) pages[i] = (int32_t)i;
  std::shuffle(pages.begin(), pages.end(), r);
  std::vector<int32_t> src(pages.begin(), pages.begin() + n * C);
  std::vector<int32_t> dst(pages.begin() + n * C, pages.begin() + 2 * n * C);
  uint8_t *sc = sh.has_scales ? scales.data() : nullptr;
  CHECK(eao_store_blocks(&sh, cache.data(), sc, tier.data(), S, src.data(), slots.data(),
                         nullptr, (int32_t)n) == 0, "store rc", -1);
  CHECK(eao_load_blocks(&sh, tier.data(), S, cache.data(), sc, slots.data(), dst.data(),
                        (int32_t)n) == 0, "load rc", -1);
  for (int64_t l = 0; l < L; ++l)
    for (int64_t i = 0; i < n * C; ++i) {
      CHECK(std::memcmp(&cache[(size_t)((l * P + dst[i]) * piece)],
                        &cache[(size_t)((l * P + src[i]) * piece)], (size_t)piece) == 0,
            "round trip", i);
      if (sc)
        CHECK(std::memcmp(&scales[(size_t)((l * P + dst[i]) * 8)],
                          &scales[(size_t)((l * P + src[i]) * 8)], 8) == 0,
              "round trip scales", i);
    }
}

}  // namespace

int main(int argc, char **argv) {
  if (argc != 3) {
    std::fprintf(stderr, "usage: %s <seed> <requests>\n", argv[0]);
    return 2;
  }
  const uint64_t seed = std::strtoull(argv[1], nullptr, 10);
  const int64_t requests = std::strtoll(argv[2], nullptr, 10);
  fuzz_tier(seed, requests);
  fuzz_stack(seed);
  fuzz_oracle_bytes(seed);
  std::printf("ok seed %llu requests %lld\n", (unsigned long long)seed, (long long)requests);
  return 0;
}
