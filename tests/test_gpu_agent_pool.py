"""GPU parity of the agent pool at its full size: 64 agents, a 64 GiB tier,
6 turns each.  Every turn's lookup, admission, allocation and the tier's full
metadata are compared with the oracle, and every loaded page is checked
against its key's pattern.

The tier is 64 GiB of pinned, device-mapped host memory.  Where the driver
caps such memory near 66 GiB per process, kernels loaded and buffers kept by
earlier GPU tests in the same process take the rest of the headroom, so this
test has a file of its own that pytest collects before the other GPU tests.
"""
import gc

import numpy as np

import oracle
import pytest
from paper_2609_33762_amd import api, drivers, workloads as W

from gpu_common import need_gpu

pytestmark = pytest.mark.gpu


def release(torch):
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def oshape_of(sh):
    return oracle.make_shape(sh.num_pages, sh.num_layers, sh.page_tokens, sh.num_kv_heads,
                             sh.head_dim, sh.elem_bytes, sh.has_scales)


def test_agent_pool_metadata_and_bytes():
    torch = need_gpu()
    sh = W.QWEN3
    kv = torch.empty(sh.cache_bytes, dtype=torch.uint8, device="cuda")
    cache = api.Cache(kv, sh.num_pages, sh.num_layers, sh.page_tokens, sh.num_kv_heads,
                      sh.head_dim, sh.elem_bytes)
    tier = api.Tier(cache, W.POOL_TIER_BYTES)
    beta = sh.num_layers * sh.piece_bytes // sh.page_tokens
    # kappa = 256 blocks: refills above 4,096 tokens are declined under pressure
    kw = dict(kappa=256, block_tokens=sh.page_tokens, activity_window=W.POOL_AGENTS)
    pol = api.make_policy(beta_rank=beta, **kw)
    opol = oracle.make_policy(beta=beta, **kw)
    ot = oracle.Tier(oshape_of(sh), W.POOL_TIER_BYTES)
    assert ot.capacity == tier.capacity == 43690
    pool = drivers.AgentPool(torch, cache, tier, kv, sh, pol)
    declined = evicted = 0
    records = []
    for t in range(6 * W.POOL_AGENTS):
        rec = pool.turn()
        records.append(rec)
        assert rec.loaded_ok, f"turn {t}: a loaded page differs from its key's pattern"
        h, hs = ot.lookup(rec.keys)
        assert h == rec.hit and np.array_equal(hs, rec.hit_slots), t
        save, mask = ot.admission(opol, rec.n_tokens, rec.hit * sh.page_tokens, rec.agent, t,
                                  rec.keys)
        assert save == rec.save and np.array_equal(mask, rec.mask), t
        _, slots = ot.alloc(rec.keys, mask)
        assert np.array_equal(slots, rec.alloc_slots), t
        ok = slots >= 0
        ot.mark_stored(slots[ok])
        if ok.any():
            ot.unpin(slots[ok])
        if h:
            ot.unpin(hs)
        declined += int(not save)
        if t % 16 == 15 or t == 6 * W.POOL_AGENTS - 1:
            a, b = tier.export(), ot.export()
            for k in ("state", "pins", "keys", "lru"):
                assert np.array_equal(a[k], b[k]), (t, k)
        sa, sb = tier.stats(), ot.stats()
        for k in ("allocated", "registered", "evictions_total", "active_tasks", "last_pressure"):
            assert sa[k] == sb[k], (t, k)
        evicted = sa["evictions_total"]
    # the run crosses the capacity transition: the tier evicts and declines refills
    assert evicted > 0 and declined > 0
    # the capacity tool on the run's own reference stream, against the oracle's
    # reference model at the tier's K_H, with and without the run's declines
    refs = np.concatenate([r.keys for r in records])
    lens = [len(r.keys) for r in records]
    dec = np.repeat([not r.save for r in records], lens).astype(np.uint8)
    prev, _ = api.reuse_distances(refs)
    full = oracle.lru_reference(refs, tier.capacity).astype(bool)
    assert np.array_equal((prev >= 0) & (prev < tier.capacity), full)
    assert np.array_equal(api.lru_simulate(refs, tier.capacity, dec),
                          oracle.lru_reference(refs, tier.capacity, dec))
    rep = drivers.stack_report(records, tier.capacity, tier.slot_bytes, [64 << 30])
    assert rep["hits_measured"] == sum(r.hit for r in records)
    # the tier's own order with the run's declines predicts every lookup
    assert np.array_equal(rep["hits_tier_order_per_request"], [r.hit for r in records])
    assert rep["references"] == len(refs) and rep["declined_new_blocks"] > 0
    tier.close()
    cache.close()
    del kv
    release(torch)
