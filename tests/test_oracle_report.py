"""Pins of the oracle's published telemetry and of the write rule driven by
a report (App. "Runtime Admission Details": the worker publishes the
registered chunks, K_H and the evictions of the last window; a decision
uses the scheduler's copy when it is fresh, and the working-set estimate
alone otherwise; Eq. 10).

* The report counts exactly the evictions the test caused inside the window.
* Truth table of the rule over (over, full, evicting, fresh/stale/none).
* A report taken at the decision's own time gives the same decisions as the
  tier's live state; a stale or missing report the same as no telemetry,
  on random operation sequences.
* Freshness boundary: age == max_age is fresh, one more is stale, and a
  report newer than the decision is ignored.
"""
import itertools

import numpy as np
import pytest

import oracle

from test_oracle_tier import BETA, N, SHAPE, SLOT, _fill, build_state, key_of


def decide_with(t, report, max_age, over, u, now=1, kappa=2, telemetry=1):
    pol = oracle.make_policy(kappa=kappa, block_tokens=1, beta=BETA, activity_window=10,
                             telemetry=telemetry)
    A = 5 if over else 4  # (A-1) * N * beta against C_H = 320 bytes
    for a in range(1, A - 1):
        t.admission(pol, N, N, task_id=a, now=now, keys=np.zeros((N, 32), np.uint8) + 7)
    keys = np.stack([key_of(7000 + i)[0] for i in range(N)])
    save, mask = t.admission_report(pol, N, N - u, A - 1, now, keys, report, max_age)
    assert t.stats()["active_tasks"] == A
    return save, mask


def test_report_counts_evictions_inside_the_window():
    K = 4
    t = oracle.Tier(SHAPE, K * SLOT)
    r = t.publish(0, 10)
    assert (r.time, r.registered, r.capacity_slots, r.evictions) == (0, 0, 4, 0)
    _fill(t, 4)                      # no eviction yet
    t.publish(2, 10)                 # the tier's clock is now 2
    _fill(t, 2, start=10)            # two evictions, stamped 2
    t.publish(5, 10)
    _fill(t, 1, start=20)            # one eviction, stamped 5
    r = t.publish(7, 3)              # window (4, 7]: the eviction at 5
    assert (r.time, r.registered, r.evictions) == (7, 4, 1)
    assert t.publish(7, 6).evictions == 3     # (1, 7]: all three
    assert t.publish(7, 2).evictions == 0     # (5, 7]: none (t > now - W)
    assert t.stats()["evictions_total"] == 3


@pytest.mark.parametrize("over,full,evicting,fresh,u",
                         list(itertools.product([0, 1], [0, 1], [0, 1],
                                                ["fresh", "stale", "none"], [2, 3])))
def test_rule_with_a_report_truth_table(over, full, evicting, fresh, u):
    t = build_state(full, evicting)
    rep = t.publish(0, 10)
    assert (rep.evictions > 0) == bool(evicting)
    report = None if fresh == "none" else rep
    max_age = 5 if fresh == "fresh" else 0          # the decision comes at time 1
    save, mask = decide_with(t, report, max_age, over, u)
    pressure = over and (fresh != "fresh" or (full and evicting))
    assert save == int(not (pressure and u > 2))
    assert mask.sum() == (N if save else 0)


def test_freshness_boundary():
    t = build_state(True, True)
    rep = t.publish(0, 10)
    # under pressure the report decides: full and evicting -> skip a refill
    s, _ = decide_with(t, rep, 3, over=True, u=3, now=3)      # age 3 == max_age: fresh
    assert s == 0
    t = build_state(False, False)
    rep = t.publish(0, 10)
    s_fresh, _ = decide_with(t, rep, 3, over=True, u=3, now=3)
    assert s_fresh == 1                                         # fresh, not full: store
    t = build_state(False, False)
    rep = t.publish(0, 10)
    s_stale, _ = decide_with(t, rep, 2, over=True, u=3, now=3)  # age 3 > 2: stale
    assert s_stale == 0                                         # the estimate alone skips
    t = build_state(False, False)
    # a report from the future saying "not full" would let the write through
    future = oracle.TierReport(5, 0, 10, 0)
    s_future, _ = decide_with(t, future, 10, over=True, u=3, now=3)
    assert s_future == 0                                        # ignored: the estimate skips
    # telemetry off in the policy: a fresh report is not used either
    t = build_state(False, False)
    rep = t.publish(0, 10)
    s_off, _ = decide_with(t, rep, 5, over=True, u=3, telemetry=0)
    assert s_off == 0


@pytest.mark.parametrize("seed", range(5))
def test_report_at_decision_time_equals_live_state(seed):
    rng = np.random.default_rng(seed)
    K = 12
    live, rep_now = oracle.Tier(SHAPE, K * SLOT), oracle.Tier(SHAPE, K * SLOT)
    none, stale = oracle.Tier(SHAPE, K * SLOT), oracle.Tier(SHAPE, K * SLOT)
    # beta = 40: C_reuse = (A-1) * Nbar * 40 crosses C_H = 384 bytes as the
    # active pool changes, and the 40-key universe keeps the 12-slot tier
    # evicting
    pol1 = oracle.make_policy(kappa=1, block_tokens=1, beta=40, activity_window=6, telemetry=1)
    pol0 = oracle.make_policy(kappa=1, block_tokens=1, beta=40, activity_window=6, telemetry=0)
    now = 0
    outcomes = {"live": set(), "none": set()}
    for step in range(160):
        now += int(rng.integers(0, 3))
        n = int(rng.integers(1, 6))
        keys = np.stack([key_of(int(c))[0] for c in rng.integers(0, 40, size=n)])
        task = int(rng.integers(0, 8))
        a = live.admission(pol1, n, 0, task, now, keys)
        b = rep_now.admission_report(pol1, n, 0, task, now, keys, rep_now.publish(now, 6), 0)
        c = none.admission(pol0, n, 0, task, now, keys)
        old = oracle.TierReport(now - 7, 0, K, 0)
        d = stale.admission_report(pol1, n, 0, task, now, keys, old, 6)
        assert a[0] == b[0] and np.array_equal(a[1], b[1]), step
        assert c[0] == d[0] and np.array_equal(c[1], d[1]), step
        outcomes["live"].add(a[0])
        outcomes["none"].add(c[0])
        # store what each tier admitted, then release the pins
        for t, (save, mask) in ((live, a), (rep_now, b), (none, c), (stale, d)):
            _, slots = t.alloc(keys, mask)
            ok = slots >= 0
            t.mark_stored(slots[ok])
            t.unpin(slots[ok])
    assert outcomes == {"live": {0, 1}, "none": {0, 1}}  # both decisions occur
    for x, y in ((live, rep_now), (none, stale)):
        ex, ey = x.export(), y.export()
        for k in ("state", "keys", "lru"):
            assert np.array_equal(ex[k], ey[k])


def test_publish_and_report_errors():
    t = oracle.Tier(SHAPE, 4 * SLOT)
    t.publish(5, 10)
    with pytest.raises(oracle.OracleError):
        t.publish(4, 10)                  # the clock does not run backwards
    with pytest.raises(oracle.OracleError):
        t.publish(6, -1)
    pol = oracle.make_policy(kappa=1, block_tokens=1, beta=1)
    with pytest.raises(oracle.OracleError):
        t.admission_report(pol, 1, 0, 0, 6, key_of(1), None, -1)
