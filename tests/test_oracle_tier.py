"""Pins of the oracle's host-tier metadata and write admission.

* Lemma 1 and Proposition 1 of the paper (App. 'Runtime Admission Details',
  'Reference model') checked on random reference streams with brute-force
  reuse distances: the oracle's LRU must satisfy both.
* The write rule of Eq. 6 / Eq. 10 checked as a truth table, including its
  endpoints p = 0 (offload) and p = 1 (fixed admission) (section 4).
* A brute-force Python model of the tier (list-based recency, linear scans)
  compared state-for-state on random operation sequences.
"""
import itertools

import numpy as np
import pytest

import oracle

SLOT = 32  # slot bytes of the tiny shape below
SHAPE = oracle.make_shape(1, 1, 1, 1, 16, 1)  # 2*1*1*16*1 = 32 B per slot


def key_of(c):
    return np.frombuffer(int(c + 1).to_bytes(32, "little"), np.uint8).reshape(1, 32)


def run_stream(stream, K, declined=frozenset()):
    """Drive the reference model through the tier: every reference is a
    one-chunk lookup; a miss inserts unless the reference is declined."""
    tier = oracle.Tier(SHAPE, K * SLOT)
    assert tier.capacity == K
    hits, promoted = [], []
    for i, c in enumerate(stream):
        h, slots = tier.lookup(key_of(c))
        if h == 1:
            tier.unpin(slots)
            hits.append(True)
            promoted.append(True)
        else:
            hits.append(False)
            if i in declined:
                promoted.append(False)
            else:
                n, s = tier.alloc(key_of(c))
                assert n == 1
                tier.mark_stored(s)
                tier.unpin(s)
                promoted.append(True)
    return hits, promoted


def next_ref(stream):
    nxt = [None] * len(stream)
    last = {}
    for i in range(len(stream) - 1, -1, -1):
        nxt[i] = last.get(stream[i])
        last[stream[i]] = i
    return nxt


def distinct_between(stream, s, t, y, keep=None):
    return len({stream[i] for i in range(s + 1, t)
                if stream[i] != y and (keep is None or keep[i])})


def random_stream(rng, universe, T):
    w = rng.dirichlet(np.full(universe, 0.6))
    return list(rng.choice(universe, size=T, p=w))


@pytest.mark.parametrize("seed", range(12))
def test_lemma1_and_proposition1(seed):
    rng = np.random.default_rng(seed)
    K = int(rng.integers(2, 7))
    stream = random_stream(rng, int(rng.integers(K + 2, 4 * K + 4)), 160)
    nxt = next_ref(stream)
    full_hits, full_prom = run_stream(stream, K)
    assert all(full_prom)
    # Lemma 1 under full admission: hit at t iff D(s,t) < K_H
    prev = {}
    for t, y in enumerate(stream):
        if y in prev:
            assert full_hits[t] == (distinct_between(stream, prev[y], t, y) < K), t
        else:
            assert not full_hits[t]
        prev[y] = t
    # restricted policy: decline a random subset of references whose next
    # reuse distance is >= K_H (or that are never referenced again)
    eligible = [i for i in range(len(stream))
                if nxt[i] is None or distinct_between(stream, i, nxt[i], stream[i]) >= K]
    declined = frozenset(i for i in eligible if rng.random() < 0.7)
    r_hits, r_prom = run_stream(stream, K, declined)
    # Proposition 1: every full-admission hit also hits
    for t in range(len(stream)):
        if full_hits[t]:
            assert r_hits[t], t
    assert sum(r_hits) >= sum(full_hits)
    # Lemma 1 under the restricted policy, with P counted over promotions
    prev = {}
    for t, y in enumerate(stream):
        if y in prev:
            s = prev[y]
            if r_prom[s]:
                P = distinct_between(stream, s, t, y, keep=r_prom)
                assert r_hits[t] == (P < K), t
                # converse: hits gained are those with P < K <= D
                if r_hits[t] and not full_hits[t]:
                    assert distinct_between(stream, s, t, y) >= K
            else:
                assert not r_hits[t]
        prev[y] = t


def test_declining_a_near_reuse_can_lose_a_hit():
    # the condition D >= K_H matters: declining a chunk that returns within
    # capacity loses its hit (App. 'Reuse distance of declined chunks')
    stream = [0, 1, 0]
    h_full, _ = run_stream(stream, 2)
    h_bad, _ = run_stream(stream, 2, frozenset([0]))
    assert h_full[2] and not h_bad[2]


# ------------------------------------------------------------ write rule

BETA = 1
N = 100


def _fill(tier, count, start=0):
    for c in range(start, start + count):
        n, s = tier.alloc(key_of(1000 + c))
        assert n == 1
        tier.mark_stored(s)
        tier.unpin(s)


def build_state(full, evicting, K=10):
    """Return a tier with the requested occupancy/eviction telemetry at clock 0."""
    t = oracle.Tier(SHAPE, K * SLOT)
    pol = oracle.make_policy(kappa=2, block_tokens=1, beta=BETA, activity_window=10,
                             mode=oracle.ADMIT_ALWAYS)
    # the set-up lookup is task 0 with n = N, so it is one of the A_t tasks
    t.admission(pol, N, N, task_id=0, now=0, keys=np.zeros((N, 32), np.uint8))
    if evicting:
        _fill(t, K + 1)              # the last insert evicts one chunk at clock 0
        if not full:
            n, s = t.alloc(key_of(5000))   # evicts another, then abandon it
            t.unpin(s)               # registered falls to K - 1 < 0.95 K
    else:
        _fill(t, K if full else K // 2)
    st = t.stats()
    assert (st["registered"] * 10**6 >= 950000 * K) == full
    assert (st["evictions_total"] > 0) == evicting
    return t


def decide(t, mode, telemetry, over, u, now=1, kappa=2):
    pol = oracle.make_policy(kappa=kappa, block_tokens=1, beta=BETA, activity_window=10,
                             mode=mode, telemetry=telemetry)
    # C_H = 10 slots * 32 B = 320 bytes; C_reuse = (A-1) * N * beta
    # tasks 0 (set-up) .. A-1 all look up N tokens inside the window
    A = 5 if over else 4            # 400 > 320, 300 < 320
    for a in range(1, A - 1):
        t.admission(pol, N, N, task_id=a, now=now, keys=np.zeros((N, 32), np.uint8) + 7)
    keys = np.stack([key_of(7000 + i)[0] for i in range(N)])
    save, mask = t.admission(pol, N, N - u, task_id=A - 1, now=now, keys=keys)
    st = t.stats()
    assert st["active_tasks"] == A and st["mean_prompt"] == N
    return save, mask


@pytest.mark.parametrize("over,full,evicting,telemetry,u",
                         list(itertools.product([0, 1], [0, 1], [0, 1], [0, 1], [2, 3])))
def test_conditioned_rule_truth_table(over, full, evicting, telemetry, u):
    t = build_state(full, evicting)
    save, mask = decide(t, oracle.ADMIT_CONDITIONED, telemetry, over, u)
    pressure = over and (not telemetry or (full and evicting))
    assert save == int(not (pressure and u > 2))
    assert mask.sum() == (N if save else 0)


def test_working_set_comparison_is_strict_and_uses_window():
    # C_reuse == C_H is not over; tasks outside the window do not count
    t = oracle.Tier(SHAPE, 10 * SLOT)
    pol = oracle.make_policy(kappa=0, block_tokens=1, beta=1, activity_window=5,
                             telemetry=0)
    keys = np.stack([key_of(i)[0] for i in range(80)])
    # tasks 0..4 at time 0 with n = 80: A = 5 -> (5-1) * 80 = 320 == C_H -> not over
    for a in range(5):
        save, _ = t.admission(pol, 80, 0, task_id=a, now=0, keys=keys)
    assert save == 1 and t.stats()["active_tasks"] == 5
    # a sixth task at time 4: A = 6 -> 400 > 320 -> over -> skip (u = 80 > 0)
    save, _ = t.admission(pol, 80, 0, task_id=5, now=4, keys=keys)
    assert save == 0
    # at time 5 the lookups at time 0 leave the window (t > now - W is required)
    save, _ = t.admission(pol, 80, 0, task_id=6, now=5, keys=keys)
    assert t.stats()["active_tasks"] == 2 and save == 1


def test_paper_working_set_against_capacity():
    # A = 16, Nbar = 33,234, beta = 24 KiB gives 11.41 GiB: over a 10 GiB tier,
    # under a 12 GiB one (section 3.2); the prompt-length window is 256
    beta = 24576
    shape = oracle.make_shape(1, 1, 1024, 1, 12, 1)  # 24 KiB slots (b = 1024 tokens, beta = 24)
    for cap_gib, want_over in [(10, True), (12, False)]:
        t = oracle.Tier(shape, cap_gib << 30)
        pol = oracle.make_policy(kappa=8, block_tokens=1024, beta=beta, activity_window=60,
                                 telemetry=0)
        n = 33234
        keys = np.zeros((n // 1024, 32), np.uint8)
        for a in range(16):
            save, _ = t.admission(pol, n, 0, task_id=a, now=1, keys=keys)
        st = t.stats()
        assert st["active_tasks"] == 16 and st["mean_prompt"] == n
        assert save == int(not want_over)  # u = 32 > kappa = 8


def test_endpoints_and_kappa_boundary():
    for u in range(0, 6):
        s_always, _ = decide(build_state(True, True), oracle.ADMIT_ALWAYS, 1, True, u, kappa=2)
        s_fixed, _ = decide(build_state(False, False), oracle.ADMIT_FIXED, 1, False, u, kappa=2)
        assert s_always == 1
        assert s_fixed == int(u <= 2)  # u > kappa is strict


def test_decision_holds_for_the_request_and_dedup():
    t = oracle.Tier(SHAPE, 8 * SLOT)
    _fill(t, 3)  # keys 1000..1002 resident
    pol = oracle.make_policy(kappa=0, block_tokens=1, beta=1, telemetry=0,
                             mode=oracle.ADMIT_FIXED)
    keys = np.stack([key_of(c)[0] for c in [1000, 1001, 77, 1002, 78]])
    save, mask = t.admission(pol, 5, 0, 1, 0, keys)
    assert save == 0 and mask.sum() == 0
    # a later lookup of the same request keeps the first decision
    save, mask = t.admission(pol, 5, 0, 1, 0, keys, decided=1)
    assert save == 1 and list(mask) == [0, 0, 1, 0, 1]
    assert t.stats()["clock"] == 0


def test_pending_allocations_are_not_registered():
    # App. 'Runtime Admission Details': a store allocates the buffers of all
    # its chunks before it registers them, so an allocation can fail while
    # fewer chunks are registered than the tier holds; the occupancy o_t of
    # Eq. 10 is the registered chunks over K_H.  A decision or report that
    # falls between another request's allocation and its store therefore
    # sees the allocation's victim gone and the new chunk not yet counted.
    K = 10
    t = build_state(full=True, evicting=False, K=K)    # 10 of 10 registered
    n, s = t.alloc(key_of(5000))                       # evicts one chunk
    assert n == 1
    st = t.stats()
    assert (st["registered"], st["allocated"], st["evictions_total"]) == (K - 1, K, 1)
    rep = t.publish(0, 10)
    assert (rep.registered, rep.capacity_slots, rep.evictions) == (K - 1, K, 1)
    # over the capacity and evicting, but o_t = 0.9 < theta = 0.95: no pressure
    save, mask = decide(t, oracle.ADMIT_CONDITIONED, 1, over=True, u=3)
    assert save == 1 and mask.sum() == N
    # the report taken in between says the same
    save, _ = t.admission_report(oracle.make_policy(kappa=2, block_tokens=1, beta=BETA,
                                                    activity_window=10),
                                 N, N - 3, 4, 1, np.stack([key_of(7000 + i)[0] for i in range(N)]),
                                 rep, 5)
    assert save == 1
    # the pending key is still deduplicated: it is not copied a second time
    pol = oracle.make_policy(kappa=2, block_tokens=1, beta=BETA, activity_window=10)
    _, mask = t.admission(pol, 3, 0, 4, 1, np.concatenate([key_of(4999), key_of(5000),
                                                             key_of(5001)]), decided=1)
    assert list(mask) == [1, 0, 1]
    # once its store is issued the chunk is registered: full and evicting
    t.mark_stored(s)
    assert t.stats()["registered"] == K and t.publish(1, 10).registered == K
    save, _ = decide(t, oracle.ADMIT_CONDITIONED, 1, over=True, u=3, now=2)
    assert save == 0
    # an abandoned allocation never counted
    t2 = build_state(full=True, evicting=False, K=K)
    n, s2 = t2.alloc(key_of(6000))
    t2.unpin(s2)
    st = t2.stats()
    assert (st["registered"], st["allocated"]) == (K - 1, K - 1)


# ------------------------------------------------ brute-force tier model

class Model:
    FREE, PENDING, RESIDENT = 0, 1, 2

    def __init__(self, K):
        self.K = K
        self.state = [0] * K
        self.pins = [0] * K
        self.keys = [None] * K
        self.order = []  # least recent first
        self.evictions = 0

    def find(self, k):
        for s in range(self.K):
            if self.keys[s] == k:
                return s
        return None

    def touch(self, s):
        self.order.remove(s)
        self.order.append(s)

    def lookup(self, ks):
        hits = []
        for k in ks:
            s = self.find(k)
            if s is None or self.state[s] != self.RESIDENT:
                break
            hits.append(s)
        for s in hits:
            self.touch(s)
            self.pins[s] += 1
        return hits

    def alloc(self, ks, mask):
        out = []
        done = False
        for k, m in zip(ks, mask):
            if not m or done or self.find(k) is not None:
                out.append(-1)
                continue
            free = [s for s in range(self.K) if self.state[s] == self.FREE]
            if free:
                s = free[0]
            else:
                victims = [v for v in self.order if self.state[v] == self.RESIDENT and self.pins[v] == 0]
                if not victims:
                    done = True
                    out.append(-1)
                    continue
                s = victims[0]
                self.order.remove(s)
                self.evictions += 1
            self.keys[s] = k
            self.state[s] = self.PENDING
            self.pins[s] += 1
            self.order.append(s)
            out.append(s)
        return out

    def mark(self, slots):
        for s in slots:
            if self.state[s] == self.PENDING:
                self.state[s] = self.RESIDENT

    def unpin(self, slots):
        for s in slots:
            self.pins[s] -= 1
            if self.pins[s] == 0 and self.state[s] == self.PENDING:
                self.state[s] = self.FREE
                self.keys[s] = None
                self.order.remove(s)


@pytest.mark.parametrize("seed", range(8))
def test_tier_matches_brute_force_model(seed):
    rng = np.random.default_rng(100 + seed)
    K = int(rng.integers(3, 12))
    t = oracle.Tier(SHAPE, K * SLOT)
    m = Model(K)
    held = []  # pinned slot lists not yet released
    for step in range(300):
        op = rng.integers(0, 4)
        if op == 0 or op == 1:
            # a request: a chain of chunk ids drawn from a small universe
            ids = [int(x) for x in rng.choice(3 * K, size=int(rng.integers(1, K + 3)), replace=False)]
            ks = [key_of(c) for c in ids]
            karr = np.concatenate(ks)
            h, slots = t.lookup(karr)
            mh = m.lookup([c for c in ids])
            assert list(slots) == mh
            mask = (rng.random(len(ids)) < 0.8).astype(np.uint8)
            cnt, got = t.alloc(karr, mask)
            want = m.alloc(ids, mask)
            assert list(got) == want and cnt == sum(1 for x in want if x >= 0)
            stored = [s for s in want if s >= 0 and rng.random() < 0.9]
            t.mark_stored(np.array(stored, np.int64))
            m.mark(stored)
            held.append(list(slots) + [s for s in want if s >= 0])
        elif op == 2 and held:
            rel = held.pop(int(rng.integers(0, len(held))))
            t.unpin(np.array(rel, np.int64))
            m.unpin(rel)
        ex = t.export()
        assert list(ex["state"]) == m.state
        assert list(ex["pins"]) == m.pins
        assert list(ex["lru"]) == m.order
        st = t.stats()
        assert st["evictions_total"] == m.evictions
        # occupancy counts stored chunks only; allocations hold keys too
        assert st["registered"] == m.state.count(Model.RESIDENT)
        assert st["allocated"] == K - m.state.count(Model.FREE)
        for s in range(K):
            if m.keys[s] is None:
                assert not ex["keys"][s].any()
            else:
                assert ex["keys"][s].tobytes() == key_of(m.keys[s]).tobytes()


def test_everything_pinned_leaves_remaining_blocks_unallocated():
    t = oracle.Tier(SHAPE, 3 * SLOT)
    karr = np.concatenate([key_of(c) for c in range(5)])
    cnt, slots = t.alloc(karr)
    assert cnt == 3 and list(slots) == [0, 1, 2, -1, -1]
    assert t.stats()["evictions_total"] == 0


def test_unpin_errors_change_nothing():
    t = oracle.Tier(SHAPE, 4 * SLOT)
    cnt, slots = t.alloc(np.concatenate([key_of(0), key_of(1)]))
    before = t.export()
    with pytest.raises(oracle.OracleError):
        t.unpin(np.array([0, 0], np.int64))   # slot 0 holds one pin only
    after = t.export()
    for k in before:
        assert np.array_equal(before[k], after[k])


def test_active_pool_counts_distinct_tasks():
    # A_t counts tasks, not lookups: one task looking up repeatedly is one task
    t = oracle.Tier(SHAPE, 10 * SLOT)
    pol = oracle.make_policy(kappa=0, block_tokens=1, beta=1, activity_window=100,
                             telemetry=0)
    keys = np.stack([key_of(i)[0] for i in range(100)])
    for now in range(6):
        save, _ = t.admission(pol, 100, 0, task_id=3, now=now, keys=keys)
    assert t.stats()["active_tasks"] == 1 and save == 1
    for a in range(4):
        save, _ = t.admission(pol, 100, 0, task_id=10 + a, now=7, keys=keys)
    # 5 distinct tasks: (5-1) * 100 = 400 > 320
    assert t.stats()["active_tasks"] == 5 and save == 0
