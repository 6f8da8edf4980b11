// Reuse-distance capacity tool (section 3.2, Eq. 4; App. "Prefix coverage
// from a reference stream").  Host-only: no HIP call.
//
// Reuse distances come from one pass over the stream with a Fenwick tree
// over reference positions that holds a 1 at the latest reference of every
// chunk seen so far.  When chunk y is referenced at i after its previous
// reference s, every distinct chunk referenced strictly between s and i
// has its latest reference in (s, i), and no other chunk does, so the tree's
// count over (s, i) is D(s, i).  The 1 then moves from s to i.  Because LRU
// holds the K most recently referenced chunks when every miss is admitted
// (Mattson's stack property), one pass answers every capacity at once:
// reference i hits in a tier of K chunks exactly when 0 <= D < K.
#include <stdint.h>

#include <algorithm>
#include <cstring>
#include <new>
#include <unordered_map>
#include <vector>

#include "ea.h"
#include "ea_tier_meta.hpp"

namespace {

// Keys passed to the tool need not be SHA-256 digests: mix all 32 bytes.
struct MixHash {
  size_t operator()(const ea::Key &k) const {
    uint64_t h = k.w[0] * 0x9E3779B97F4A7C15ull;
    h ^= (k.w[1] + (h << 6) + (h >> 2)) * 0xC2B2AE3D27D4EB4Full;
    h ^= (k.w[2] + (h << 6) + (h >> 2)) * 0x165667B19E3779F9ull;
    h ^= (k.w[3] + (h << 6) + (h >> 2)) * 0x9E3779B97F4A7C15ull;
    return (size_t)(h ^ (h >> 29));
  }
};

// Counts over positions 0..n-1 with point updates and prefix sums.
class Fenwick {
 public:
  explicit Fenwick(int64_t n) : t_((size_t)n + 1, 0) {}
  void add(int64_t i, int64_t v) {
    for (int64_t x = i + 1; x < (int64_t)t_.size(); x += x & -x) t_[(size_t)x] += v;
  }
  // sum over positions 0..i-1
  int64_t prefix(int64_t i) const {
    int64_t s = 0;
    for (int64_t x = i; x > 0; x -= x & -x) s += t_[(size_t)x];
    return s;
  }

 private:
  std::vector<int64_t> t_;
};

}  // namespace

extern "C" int ea_reuse_distances(const uint8_t *refs, int64_t n, int64_t *prev_dist,
                                  int64_t *next_dist) {
  if (n < 0 || (n > 0 && refs == nullptr)) return EA_EINVAL;
  if (n == 0) return EA_OK;
  try {
    std::vector<int64_t> prev((size_t)n), next((size_t)n, -1);
    std::unordered_map<ea::Key, int64_t, MixHash> latest;
    latest.reserve((size_t)std::min<int64_t>(n, (int64_t)1 << 26));
    Fenwick marks(n);
    for (int64_t i = 0; i < n; ++i) {
      auto ins = latest.try_emplace(ea::Key::from(refs + 32 * i), i);
      if (ins.second) {
        prev[(size_t)i] = -1;
      } else {
        const int64_t s = ins.first->second;
        const int64_t d = marks.prefix(i) - marks.prefix(s + 1);
        prev[(size_t)i] = d;
        next[(size_t)s] = d;
        marks.add(s, -1);
        ins.first->second = i;
      }
      marks.add(i, 1);
    }
    if (prev_dist) std::memcpy(prev_dist, prev.data(), (size_t)n * sizeof(int64_t));
    if (next_dist) std::memcpy(next_dist, next.data(), (size_t)n * sizeof(int64_t));
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
  return EA_OK;
}

extern "C" int ea_prefix_coverage(const int64_t *prev_dist, const int64_t *req_off,
                                  int64_t n_req, const int64_t *caps, int64_t n_caps,
                                  int64_t *coverage) {
  if (n_req < 0 || n_caps < 0 || req_off == nullptr) return EA_EINVAL;
  if (n_req > 0 && n_caps > 0 && coverage == nullptr) return EA_EINVAL;
  if (n_caps > 0 && caps == nullptr) return EA_EINVAL;
  if (req_off[0] < 0) return EA_EINVAL;
  for (int64_t j = 0; j < n_req; ++j)
    if (req_off[j + 1] < req_off[j]) return EA_EINVAL;
  for (int64_t c = 0; c < n_caps; ++c)
    if (caps[c] < 0) return EA_EINVAL;
  if (req_off[n_req] > req_off[0] && prev_dist == nullptr) return EA_EINVAL;
  int64_t longest = 0;
  for (int64_t j = 0; j < n_req; ++j) longest = std::max(longest, req_off[j + 1] - req_off[j]);
  try {
    // running maximum of a request's distances (allocated before any output
    // is written, so an allocation failure leaves coverage untouched)
    std::vector<int64_t> run((size_t)longest);
    for (int64_t j = 0; j < n_req; ++j) {
      const int64_t b = req_off[j], len = req_off[j + 1] - b;
      int64_t m = -1;
      for (int64_t i = 0; i < len; ++i) {
        const int64_t d = prev_dist[b + i];
        // a first reference misses at every capacity
        m = std::max(m, d < 0 ? INT64_MAX : d);
        run[(size_t)i] = m;
      }
      // leading hits at capacity K: references before the first running
      // maximum >= K
      for (int64_t c = 0; c < n_caps; ++c)
        coverage[j * n_caps + c] =
            std::lower_bound(run.begin(), run.begin() + len, caps[c]) - run.begin();
    }
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
  return EA_OK;
}

// The reference model itself for one capacity, with declined misses: the
// one-pass distances above cover full admission only, because which
// references promote a chunk then depends on the capacity.  Recency is an
// intrusive list over at most K entries, linked by index.
extern "C" int ea_lru_simulate(const uint8_t *refs, int64_t n, const uint8_t *declined,
                               int64_t capacity, uint8_t *hits) {
  if (n < 0 || capacity < 0 || (n > 0 && (refs == nullptr || hits == nullptr)))
    return EA_EINVAL;
  if (n == 0) return EA_OK;
  try {
    const int64_t k = std::min(capacity, n);
    std::vector<uint8_t> out((size_t)n, 0);
    std::vector<ea::Key> key((size_t)k);
    std::vector<int64_t> up((size_t)k, -1), down((size_t)k, -1);  // toward newer / older
    std::unordered_map<ea::Key, int64_t, MixHash> where;
    where.reserve((size_t)k);
    int64_t newest = -1, oldest = -1, used = 0;
    auto detach = [&](int64_t e) {
      if (up[(size_t)e] >= 0) down[(size_t)up[(size_t)e]] = down[(size_t)e]; else newest = down[(size_t)e];
      if (down[(size_t)e] >= 0) up[(size_t)down[(size_t)e]] = up[(size_t)e]; else oldest = up[(size_t)e];
    };
    auto make_newest = [&](int64_t e) {
      up[(size_t)e] = -1;
      down[(size_t)e] = newest;
      if (newest >= 0) up[(size_t)newest] = e;
      newest = e;
      if (oldest < 0) oldest = e;
    };
    for (int64_t i = 0; i < n && k > 0; ++i) {
      const ea::Key x = ea::Key::from(refs + 32 * i);
      auto it = where.find(x);
      if (it != where.end()) {
        out[(size_t)i] = 1;
        detach(it->second);
        make_newest(it->second);
        continue;
      }
      if (declined != nullptr && declined[i]) continue;
      int64_t e;
      if (used < k) {
        e = used++;
      } else {
        e = oldest;
        detach(e);
        where.erase(key[(size_t)e]);
      }
      key[(size_t)e] = x;
      where.emplace(x, e);
      make_newest(e);
    }
    std::memcpy(hits, out.data(), (size_t)n);
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
  return EA_OK;
}

// The tier's own order, request by request: the lookup promotes only the
// leading resident chunks, so chunks resident after the first miss keep
// their age (unlike the reference model, where every reference promotes).
// Insertions are decided before any is made (copy-time deduplication) and
// the request's own chunks are pinned against eviction until it ends.
extern "C" int ea_lru_simulate_prefix(const uint8_t *refs, const int64_t *req_off,
                                      int64_t n_req, const uint8_t *declined,
                                      int64_t capacity, int64_t *hit_blocks) {
  if (n_req < 0 || capacity < 0 || req_off == nullptr) return EA_EINVAL;
  if (n_req > 0 && hit_blocks == nullptr) return EA_EINVAL;
  if (req_off[0] != 0) return EA_EINVAL;
  int64_t longest = 0;
  for (int64_t j = 0; j < n_req; ++j) {
    if (req_off[j + 1] < req_off[j]) return EA_EINVAL;
    longest = std::max(longest, req_off[j + 1] - req_off[j]);
  }
  const int64_t n = req_off[n_req];
  if (n > 0 && refs == nullptr) return EA_EINVAL;
  try {
    const int64_t k = std::min(capacity, n);
    std::vector<int64_t> out((size_t)n_req, 0);
    std::vector<ea::Key> key((size_t)k);
    std::vector<int64_t> up((size_t)k, -1), down((size_t)k, -1), owner((size_t)k, -1);
    std::vector<int64_t> todo;
    todo.reserve((size_t)longest);
    std::unordered_map<ea::Key, int64_t, MixHash> where;
    where.reserve((size_t)k);
    int64_t newest = -1, oldest = -1, used = 0;
    auto detach = [&](int64_t e) {
      if (up[(size_t)e] >= 0) down[(size_t)up[(size_t)e]] = down[(size_t)e]; else newest = down[(size_t)e];
      if (down[(size_t)e] >= 0) up[(size_t)down[(size_t)e]] = up[(size_t)e]; else oldest = up[(size_t)e];
    };
    auto make_newest = [&](int64_t e) {
      up[(size_t)e] = -1;
      down[(size_t)e] = newest;
      if (newest >= 0) up[(size_t)newest] = e;
      newest = e;
      if (oldest < 0) oldest = e;
    };
    for (int64_t j = 0; j < n_req && k > 0; ++j) {
      const uint8_t *r = refs + 32 * req_off[j];
      const int64_t len = req_off[j + 1] - req_off[j];
      int64_t h = 0;
      for (; h < len; ++h) {
        auto it = where.find(ea::Key::from(r + 32 * h));
        if (it == where.end()) break;
        detach(it->second);
        make_newest(it->second);
        owner[(size_t)it->second] = j;
      }
      out[(size_t)j] = h;
      if (declined != nullptr && declined[j]) continue;
      todo.clear();
      for (int64_t i = h; i < len; ++i)
        if (where.find(ea::Key::from(r + 32 * i)) == where.end()) todo.push_back(i);
      for (int64_t i : todo) {
        const ea::Key x = ea::Key::from(r + 32 * i);
        if (where.count(x)) continue;  // repeated within the request
        int64_t e;
        if (used < k) {
          e = used++;
        } else {
          e = oldest;  // the request's own chunks sit at the newer end
          while (e >= 0 && owner[(size_t)e] == j) e = up[(size_t)e];
          if (e < 0) continue;
          detach(e);
          where.erase(key[(size_t)e]);
        }
        key[(size_t)e] = x;
        owner[(size_t)e] = j;
        where.emplace(x, e);
        make_newest(e);
      }
    }
    if (n_req > 0) std::memcpy(hit_blocks, out.data(), (size_t)n_req * sizeof(int64_t));
  } catch (const std::bad_alloc &) {
    return EA_ENOMEM;
  }
  return EA_OK;
}
