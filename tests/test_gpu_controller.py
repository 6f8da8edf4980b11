"""GPU tests of the write-admission controller (App. "Runtime Admission
Details"; Table "Write-admission parameters").

* Manual clock: the controller's reports, its scheduler copy and every
  decision, allocation and lookup on a random request stream equal the
  oracle driven through the same schedule (publish every report interval,
  read every read interval, a publish before a read at equal times, decide
  with the copy when fresh), including stale copies.
* Steady clock: the publisher thread runs, the copy is fresh, a decision
  uses it; before the first report the working-set estimate alone decides;
  destroying the controller joins its thread at once.
"""
import time

import numpy as np
import pytest

import oracle
from paper_2609_33762_amd import _native as N, api, workloads as W

from gpu_common import need_gpu

pytestmark = pytest.mark.gpu

SH = W.TINY
B = SH.page_tokens


def key_of(c):
    return np.frombuffer(int(c + 1).to_bytes(32, "little"), np.uint8)


def make_tier(torch, K):
    kv = torch.empty(SH.cache_bytes, dtype=torch.uint8, device="cuda")
    W.fill_bf16_normal(kv, 5)
    cache = api.Cache(kv, SH.num_pages, SH.num_layers, SH.page_tokens, SH.num_kv_heads,
                      SH.head_dim, SH.elem_bytes)
    slot = SH.num_layers * SH.piece_bytes
    tier = api.Tier(cache, K * slot)
    assert tier.capacity == K
    return kv, cache, tier, slot


class OracleSchedule:
    """The paper's schedule on the oracle tier."""

    def __init__(self, ot, pol, ri, rd, max_age, window):
        self.ot, self.pol = ot, pol
        self.ri, self.rd, self.max_age, self.window = ri, rd, max_age, window
        self.next_pub, self.next_read, self.now = ri, rd, 0
        self.hist, self.seen = [], None

    def advance(self, now):
        while min(self.next_pub, self.next_read) <= now:
            if self.next_pub <= self.next_read:
                self.hist.append(self.ot.publish(self.next_pub, self.window))
                self.next_pub += self.ri
            else:
                older = [r for r in self.hist if r.time <= self.next_read]
                if older:
                    self.seen = older[-1]
                self.next_read += self.rd
        self.now = now

    def decide(self, n, h, task, keys):
        return self.ot.admission_report(self.pol, n, h, task, self.now, keys, self.seen,
                                        self.max_age)


def fields(r):
    return (r.time, r.registered, r.capacity_slots, r.evictions) if not isinstance(r, dict) \
        else (r["time"], r["registered"], r["capacity_slots"], r["evictions"])


@pytest.mark.parametrize("seed", [0, 1])
def test_manual_clock_matches_oracle_schedule(seed):
    torch = need_gpu()
    K = 24
    kv, cache, tier, slot = make_tier(torch, K)
    beta = slot // B
    ri, rd, max_age, window = 1_000_000, 500_000, 1_200_000, 6_000_000
    kw = dict(kappa=2, block_tokens=B)
    pol = api.make_policy(beta_rank=beta, activity_window=1, **kw)  # window set by the controller
    ctl = api.Controller(tier, pol, ri, rd, max_age, window, manual_clock=True)
    ot = oracle.Tier(oracle.make_shape(SH.num_pages, SH.num_layers, SH.page_tokens,
                                       SH.num_kv_heads, SH.head_dim, SH.elem_bytes), K * slot)
    sched = OracleSchedule(ot, oracle.make_policy(beta=beta, activity_window=window, **kw),
                           ri, rd, max_age, window)
    r = np.random.default_rng(seed)
    now = 0
    saves = set()
    for step in range(300):
        now += int(r.integers(0, 900_000))
        ctl.advance(now)
        sched.advance(now)
        task = int(r.integers(0, 10))
        nb = int(r.integers(1, 9))
        keys = np.stack([key_of(task * 100 + int(c)) for c in
                         np.sort(r.choice(12, size=nb, replace=False))])
        h, hs = tier.lookup(keys)
        oh, ohs = ot.lookup(keys)
        assert h == oh and np.array_equal(hs, ohs), step
        save, mask = ctl.decide(nb * B, h * B, task, keys)
        osave, omask = sched.decide(nb * B, h * B, task, keys)
        assert save == osave and np.array_equal(mask, omask), step
        saves.add(save)
        _, slots = tier.alloc(keys, mask)
        _, oslots = ot.alloc(keys, omask)
        assert np.array_equal(slots, oslots), step
        ok = slots >= 0
        if ok.any():
            pages = W.distinct(r, SH.num_pages, int(ok.sum()))
            tier.store(cache, pages, slots[ok])
            ot.mark_stored(slots[ok])
            tier.unpin(slots[ok])
            ot.unpin(oslots[ok])
        if h:
            tier.unpin(hs)
            ot.unpin(ohs)
        st = ctl.status()
        assert st["now"] == now and st["reports_published"] == len(sched.hist), step
        if sched.hist:
            assert fields(st["published"]) == fields(sched.hist[-1]), step
        assert bool(st["have_seen"]) == (sched.seen is not None)
        if sched.seen is not None:
            assert fields(st["seen"]) == fields(sched.seen), step
    st = ctl.status()
    # the stream saw both decisions, and fresh as well as stale copies
    assert saves == {0, 1}
    assert 0 < st["fresh_decisions"] < st["decisions"] == 300
    ctl.close()
    torch.cuda.synchronize()
    tier.close()
    cache.close()


def pool_requests(ctl, tasks=10, n_blocks=8):
    """First lookups of `tasks` tasks, n_blocks new blocks each; returns the
    save decisions."""
    out = []
    for task in range(tasks):
        keys = np.stack([key_of(1000 * task + i) for i in range(n_blocks)])
        out.append(ctl.decide(n_blocks * B, 0, task, keys)[0])
    return out


def test_steady_clock_publishes_and_decides_with_fresh_reports():
    torch = need_gpu()
    kv, cache, tier, slot = make_tier(torch, 24)
    pol = api.make_policy(kappa=2, block_tokens=B, beta_rank=slot // B)
    ctl = api.Controller(tier, pol, report_interval=20_000, read_interval=10_000,
                         max_report_age=500_000, window=2_000_000)
    time.sleep(0.25)
    st = ctl.status()
    assert st["reports_published"] >= 3 and st["have_seen"] and st["fresh"]
    assert st["published"]["capacity_slots"] == 24 and st["published"]["evictions"] == 0
    # fresh reports of an empty tier: not full, so every write goes through
    assert pool_requests(ctl) == [1] * 10
    st = ctl.status()
    assert st["fresh_decisions"] == st["decisions"] == 10 and st["skips"] == 0
    t0 = time.perf_counter()
    ctl.close()
    assert time.perf_counter() - t0 < 1.0
    tier.close()
    cache.close()


def test_steady_clock_without_a_report_uses_the_estimate_alone():
    torch = need_gpu()
    kv, cache, tier, slot = make_tier(torch, 24)
    pol = api.make_policy(kappa=2, block_tokens=B, beta_rank=slot // B)
    # the first report is due after 60 s: no decision here has a fresh copy
    ctl = api.Controller(tier, pol, report_interval=60_000_000, read_interval=30_000_000,
                         max_report_age=5_000_000, window=2_000_000)
    saves = pool_requests(ctl)
    # C_reuse = (A-1) * 128 tokens * 1 KiB against C_H = 24 * 16 KiB: equal at
    # A = 4 (not over: the comparison is strict), over from A = 5 on, where
    # the estimate alone declines the 8-block refills (u = 8 > kappa = 2)
    assert saves == [1, 1, 1, 1, 0, 0, 0, 0, 0, 0]
    st = ctl.status()
    assert st["reports_published"] == 0 and not st["have_seen"]
    assert st["fresh_decisions"] == 0 and st["skips"] == 6
    # the tier refuses to go while the controller is attached, and the
    # binding keeps its handle then
    assert N.load().ea_tier_destroy(tier._h) == N.EA_EINVAL
    with pytest.raises(N.EAError):
        tier.close()
    assert tier._h
    t0 = time.perf_counter()
    ctl.close()  # the publisher waits on a 60 s tick: closing must not wait for it
    assert time.perf_counter() - t0 < 1.0
    tier.close()
    assert not tier._h
    cache.close()


def test_controller_collected_with_its_tier_frees_the_tier():
    # a tier and its controller dropped together in one reference cycle:
    # whichever finaliser runs first, the tier is freed once the controller
    # is gone
    torch = need_gpu()
    kv, cache, tier, slot = make_tier(torch, 24)
    pol = api.make_policy(kappa=2, block_tokens=B, beta_rank=slot // B)
    ctl = api.Controller(tier, pol, manual_clock=True)
    tier._cycle = ctl
    handle = tier._h.value
    tier._orphaned = False
    tier.__del__()  # the tier's finaliser first: the controller still holds it
    assert tier._orphaned and tier._h.value == handle
    ctl.close()
    assert not tier._h
    del tier._cycle
    cache.close()


def test_tier_keeps_the_steady_clock_until_the_last_controller_detaches():
    # two wall-clock controllers on one tier: closing one leaves the other's
    # steady clock in place (an allocation then stamps the tier with the
    # steady clock); closing both returns the tier to the caller's clock
    torch = need_gpu()
    kv, cache, tier, slot = make_tier(torch, 8)
    pol = api.make_policy(kappa=2, block_tokens=B, beta_rank=slot // B)
    cfg = dict(report_interval=60_000_000, read_interval=30_000_000,
               max_report_age=5_000_000, window=2_000_000)
    a = api.Controller(tier, pol, **cfg)
    b = api.Controller(tier, pol, **cfg)
    a.close()
    before = time.monotonic_ns() // 1000  # the steady clock, in microseconds
    tier.alloc(key_of(1)[None, :])
    assert tier.stats()["clock"] >= before
    b.close()
    clock = tier.stats()["clock"]
    time.sleep(0.01)
    tier.alloc(key_of(2)[None, :])
    assert tier.stats()["clock"] == clock
    tier.close()
    cache.close()
