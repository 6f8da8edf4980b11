"""Parity of the library's host-tier metadata and write admission with the
oracle: random request streams through lookup / admission / alloc / store /
unpin, compared state for state (slot states, pins, keys, LRU order,
telemetry) after every step."""
import numpy as np
import pytest

import oracle
from paper_2609_33762_amd import api
from paper_2609_33762_amd import _native as N
from paper_2609_33762_amd import workloads as W

from gpu_common import Pair

pytestmark = pytest.mark.gpu

STAT_KEYS = ["capacity_slots", "allocated", "registered", "pinned", "evictions_total",
             "evictions_window", "clock", "active_tasks", "last_pressure", "last_save"]


def compare(prod, orc, where):
    a, b = prod.export(), orc.export()
    for k in ("state", "pins", "keys", "lru"):
        assert np.array_equal(a[k], b[k]), f"{where}: {k}"
    sa, sb = prod.stats(), orc.stats()
    for k in STAT_KEYS:
        assert sa[k] == sb[k], f"{where}: {k} {sa[k]} != {sb[k]}"


@pytest.mark.parametrize("mode,telemetry,seed", [
    (N.EA_ADMIT_CONDITIONED, 1, 0), (N.EA_ADMIT_CONDITIONED, 0, 1),
    (N.EA_ADMIT_ALWAYS, 1, 2), (N.EA_ADMIT_FIXED, 1, 3), (N.EA_ADMIT_CONDITIONED, 1, 4)])
def test_random_request_streams(mode, telemetry, seed):
    K = 48
    p = Pair(64, 2, 16, 1, 32, 2, K, seed=seed)  # 4 KiB slots
    beta = 2 * 2 * 32 * 2  # bytes per token of this shape
    ot = oracle.Tier(p.oshape, K * p.sizes["slot"])
    pol_p = api.make_policy(kappa=3, block_tokens=16, beta_rank=beta, activity_window=12,
                            length_window=16, mode=mode, telemetry=telemetry)
    pol_o = oracle.make_policy(kappa=3, block_tokens=16, beta=beta, activity_window=12,
                               length_window=16, mode=mode, telemetry=telemetry)
    r = W.rng(100 + seed)
    agents = [W.tokens(1000 * seed + a, 16 * 40) for a in range(6)]
    lengths = [int(r.integers(2, 10)) * 16 for _ in range(6)]
    for turn in range(60):
        a = int(r.integers(0, 6))
        lengths[a] = min(lengths[a] + int(r.integers(0, 5)) * 16 + int(r.integers(0, 16)), 16 * 40)
        if r.random() < 0.1:  # an early edit rekeys the rest of the prompt
            agents[a] = agents[a].copy()
            agents[a][int(r.integers(0, lengths[a]))] += 1
        toks = agents[a][:lengths[a]]
        keys, _ = api.hash_blocks(toks, np.array([0, len(toks)]), 16)
        h, hs = p.tier.lookup(keys)
        oh, ohs = ot.lookup(keys)
        assert h == oh and np.array_equal(hs, ohs)
        compare(p.tier, ot, f"turn {turn} lookup")
        save, mask = p.tier.admission(pol_p, len(toks), 16 * h, a, turn, keys)
        osave, omask = ot.admission(pol_o, len(toks), 16 * h, a, turn, keys)
        assert save == osave and np.array_equal(mask, omask), turn
        cnt, slots = p.tier.alloc(keys, mask)
        ocnt, oslots = ot.alloc(keys, mask)
        assert cnt == ocnt and np.array_equal(slots, oslots), turn
        got = slots >= 0
        if got.any():
            pages = W.distinct(r, 64, int(got.sum()))
            if r.random() < 0.9:
                p.tier.store(p.cache, pages, slots[got])
                ot.mark_stored(slots[got])
            rel = slots[got]
            p.tier.unpin(rel)
            ot.unpin(rel)
        if h and r.random() < 0.8:
            p.tier.unpin(hs)
            ot.unpin(ohs)
        compare(p.tier, ot, f"turn {turn}")
    p.close()


def test_all_pinned_tier_reports_unallocated_blocks():
    p = Pair(16, 1, 16, 1, 32, 2, 4, seed=1)
    keys = np.stack([np.frombuffer(int(i + 1).to_bytes(32, "little"), np.uint8) for i in range(6)])
    cnt, slots = p.tier.alloc(keys)
    assert cnt == 4 and list(slots) == [0, 1, 2, 3, -1, -1]
    assert p.tier.stats()["evictions_total"] == 0
    with pytest.raises(N.EAError):
        p.tier.unpin([0, 0])
    p.close()


def test_long_stream_with_bounded_history_matches_the_oracle():
    # More first lookups and more evictions than the tier keeps whole
    # (65,536): the library then drops history no window can reach again,
    # the oracle keeps all of it; every decision, report and statistic must
    # still agree.
    K = 8
    p = Pair(64, 1, 16, 1, 32, 2, K, seed=7)  # 2 KiB slots
    beta = 2 * 32 * 2
    ot = oracle.Tier(p.oshape, K * p.sizes["slot"])
    kw = dict(kappa=1, block_tokens=16, activity_window=12, length_window=16,
              mode=N.EA_ADMIT_CONDITIONED, telemetry=1)
    pol_p = api.make_policy(beta_rank=beta, **kw)
    pol_o = oracle.make_policy(beta=beta, **kw)
    r = W.rng(77)
    n_req = 80_000
    nblocks = np.where(r.random(n_req) < 0.05, 3, 1)
    repeat = r.random(n_req) < 0.1
    pages = r.integers(0, 64, size=n_req)
    serial = 0
    recent = []
    for t in range(n_req):
        nb = int(nblocks[t])
        if repeat[t] and recent:
            keys = recent[-1 - t % len(recent)]  # one of the last requests again
            nb = keys.shape[0]
        else:
            keys = np.zeros((nb, 32), np.uint8)
            for j in range(nb):
                serial += 1
                keys[j, :8] = np.frombuffer(serial.to_bytes(8, "little"), np.uint8)
        recent.append(keys)
        recent = recent[-4:]
        h, hs = p.tier.lookup(keys)
        oh, ohs = ot.lookup(keys)
        assert h == oh and np.array_equal(hs, ohs), t
        save, mask = p.tier.admission(pol_p, 16 * nb, 16 * h, t % 40, t, keys)
        osave, omask = ot.admission(pol_o, 16 * nb, 16 * h, t % 40, t, keys)
        assert save == osave and np.array_equal(mask, omask), t
        cnt, slots = p.tier.alloc(keys, mask)
        ocnt, oslots = ot.alloc(keys, mask)
        assert cnt == ocnt and np.array_equal(slots, oslots), t
        got = slots >= 0
        if got.any():
            p.tier.store(p.cache, np.full(int(got.sum()), pages[t]), slots[got])
            ot.mark_stored(slots[got])
            p.tier.unpin(slots[got])
            ot.unpin(slots[got])
        if h:
            p.tier.unpin(hs)
            ot.unpin(ohs)
        if t % 997 == 0 or t == n_req - 1:
            rp, ro = p.tier.publish(t, 12), ot.publish(t, 12)
            assert (rp.registered, rp.capacity_slots, rp.evictions) == \
                (ro.registered, ro.capacity_slots, ro.evictions), t
            compare(p.tier, ot, f"request {t}")
    st = p.tier.stats()
    assert st["evictions_total"] > 65_536
    p.close()


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_decisions_between_alloc_and_store(seed):
    # App. 'Runtime Admission Details': a store allocates its chunks' buffers
    # before it registers them, so the occupancy o_t counts stored chunks
    # only.  Requests here allocate, then other requests look up, decide and
    # publish before the first one's store is issued (on the GPU, through
    # ea_store_blocks); every decision, report, statistic and metadata image
    # must equal the oracle's, and a decision must differ from what counting
    # the pending allocations would give at least once.
    K = 10
    p = Pair(64, 2, 16, 1, 32, 2, K, seed=seed)  # 4 KiB slots
    ot = oracle.Tier(p.oshape, K * p.sizes["slot"])
    beta = 2 * 2 * 32 * 2
    kw = dict(kappa=0, block_tokens=16, activity_window=1000, length_window=64,
              mode=N.EA_ADMIT_CONDITIONED, telemetry=1)
    pol_p = api.make_policy(beta_rank=beta, **kw)
    pol_o = oracle.make_policy(beta=beta, **kw)
    r = W.rng(300 + seed)
    serial = [0]

    def fresh(nb):
        keys = np.zeros((nb, 32), np.uint8)
        for j in range(nb):
            serial[0] += 1
            keys[j, :8] = np.frombuffer(serial[0].to_bytes(8, "little"), np.uint8)
        return keys

    pending = []  # (keys, slots) allocated, store not issued yet
    differs = 0
    for t in range(200):
        keys = fresh(int(r.integers(1, 3)))
        nb = len(keys)
        h, hs = p.tier.lookup(keys)
        oh, ohs = ot.lookup(keys)
        assert h == oh and np.array_equal(hs, ohs), t
        st = ot.stats()
        full_alloc = st["allocated"] * 10**6 >= 950000 * K
        full_reg = st["registered"] * 10**6 >= 950000 * K
        save, mask = p.tier.admission(pol_p, 16 * nb, 16 * h, t % 8, t, keys)
        osave, omask = ot.admission(pol_o, 16 * nb, 16 * h, t % 8, t, keys)
        assert save == osave and np.array_equal(mask, omask), t
        after = ot.stats()
        over = after["working_set"] > K * p.sizes["slot"]
        differs += int(over and full_alloc and not full_reg and after["evictions_window"] > 0)
        cnt, slots = p.tier.alloc(keys, mask)
        ocnt, oslots = ot.alloc(keys, mask)
        assert cnt == ocnt and np.array_equal(slots, oslots), t
        got = slots[slots >= 0]
        if len(got):
            pending.append(got)
        rp, ro = p.tier.publish(t, 1000), ot.publish(t, 1000)
        assert (rp.registered, rp.capacity_slots, rp.evictions) == \
            (ro.registered, ro.capacity_slots, ro.evictions), t
        # issue the stores of some earlier allocations, later than their alloc
        while pending and (len(pending) > 3 or r.random() < 0.3):
            sl = pending.pop(0)
            p.tier.store(p.cache, W.distinct(r, 64, len(sl)), sl)
            ot.mark_stored(sl)
            p.tier.unpin(sl)
            ot.unpin(sl)
        if h:
            p.tier.unpin(hs)
            ot.unpin(ohs)
        compare(p.tier, ot, f"request {t}")
    assert differs > 0, "no decision fell where pending allocations matter"
    p.close()
