"""GPU parity at the workloads' full sizes, on complete images.

Every written slot and every written page is compared with the oracle's
result, byte for byte; the whole cache is snapshotted in HBM before the
operation, and afterwards only destination pages may differ; host slots
that nothing writes are poisoned beforehand and must keep the poison.

* One Qwen3-30B-A3B turn (20,000-page cache, 16 GiB tier, 2,000 pages stored,
  1,500 loaded at the same time on two streams), both transfer plans.
* The HBM gather and scatter of 2,000 pages in one launch each, as measured.
* Layer-pipelined fp8 prefix load (64k tokens = 4,096 pages, 48 layers,
  per-page scales), also on one TP8 rank's share: a consumer stream
  snapshots each layer right after its event, and each snapshot must
  already hold the layer's final bytes.
* Dense scattered batches (4,096-page cache, 4,096-slot tier, 10,000 calls of
  1-8 non-adjacent pages): the oracle replays every call on full host images
  and the final cache and tier images must be equal byte for byte.
* Agent pool on two streams and in 1,024-token chunks (the 64 GiB pool
  itself is in test_gpu_agent_pool.py).
* The longest context of the serving configuration (262,144 tokens) as one
  TP8 rank's prefix: 16,384 pages stored to shuffled slots and loaded back.
"""
import gc

import numpy as np
import pytest

import oracle
from paper_2609_33762_amd import api, drivers, _native as N, workloads as W

from gpu_common import (POISON, assert_poisoned_except, assert_rows_equal, changed_pages,
                        need_gpu, oracle_pages, oracle_slots, pages_to_host, poison_tier)

pytestmark = pytest.mark.gpu


def release(torch):
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def oshape_of(sh, num_pages=None):
    return oracle.make_shape(num_pages or sh.num_pages, sh.num_layers, sh.page_tokens,
                             sh.num_kv_heads, sh.head_dim, sh.elem_bytes, sh.has_scales)


@pytest.mark.parametrize("plan", ["direct", "staged"])
def test_qwen3_turn_full_size(plan):
    torch = need_gpu()
    sh = W.QWEN3
    L, P, piece = sh.num_layers, sh.num_pages, sh.piece_bytes
    kv = torch.empty(sh.cache_bytes, dtype=torch.uint8, device="cuda")
    W.fill_bf16_normal(kv, W.SEED_DATA)
    kv3 = kv.view(L, P, piece)
    cache = api.Cache(kv, P, L, sh.page_tokens, sh.num_kv_heads, sh.head_dim, sh.elem_bytes)
    tier = api.Tier(cache, W.QWEN3_TIER_BYTES)
    tier.set_plan(N.EA_DIR_BOTH, N.EA_PLAN_DIRECT if plan == "direct" else N.EA_PLAN_STAGED)
    r = W.rng(W.SEED_IDS)
    n_l, n_s = W.QWEN3_LOAD_PAGES, W.QWEN3_STORE_PAGES
    prefix_pages = W.distinct(r, P, n_l)
    store_pages = W.distinct(r, P, n_s, exclude=prefix_pages)
    dst = W.distinct(r, P, n_l, exclude=np.concatenate([prefix_pages, store_pages]))
    host = tier.host_view()
    poison_tier(host)  # every slot, so that any stray write shows

    toks = W.tokens(W.SEED_TOKENS, n_l * sh.page_tokens)
    pkeys, _ = api.hash_blocks(toks, np.array([0, len(toks)]), sh.page_tokens)
    cnt, pslots = tier.alloc(pkeys)
    assert cnt == n_l and list(pslots) == list(range(n_l))
    tier.store(cache, prefix_pages, pslots)
    tier.unpin(pslots)
    rkeys = W.rng(7).integers(0, 256, size=(n_s, 32), dtype=np.uint8)
    cnt, sslots = tier.alloc(rkeys)
    assert cnt == n_s
    torch.cuda.synchronize()
    before = kv.clone()  # the whole 29 GiB cache, kept in HBM
    s_store, s_load = torch.cuda.Stream(), torch.cuda.Stream()
    h, hslots = tier.lookup(pkeys)
    assert h == n_l
    tier.load(cache, hslots, dst, stream=s_load)
    tier.store(cache, store_pages, sslots, stream=s_store)
    torch.cuda.synchronize()
    tier.unpin(sslots)
    tier.unpin(hslots)

    # every written slot is the oracle's store of its source page
    want_p = oracle_slots(sh, pages_to_host(torch, kv3, prefix_pages))
    assert_rows_equal(host[pslots], want_p, "prefix slots")
    want_s = oracle_slots(sh, pages_to_host(torch, kv3, store_pages))
    assert_rows_equal(host[sslots], want_s, "refill slots")
    del want_s
    # every loaded page is the oracle's load of the oracle's slot image
    want_l = oracle_pages(sh, want_p)
    got_l = pages_to_host(torch, kv3, dst)
    assert_rows_equal(got_l.transpose(1, 0, 2), want_l.transpose(1, 0, 2), "loaded pages")
    del want_l, got_l, want_p
    # nothing else in HBM changed, and every slot nobody wrote kept its poison
    changed = changed_pages(torch, kv3, before.view(L, P, piece))
    assert np.isin(changed, dst).all(), np.setdiff1d(changed, dst)[:8]
    del before
    assert_poisoned_except(host, np.concatenate([pslots, sslots]))
    tier.close()
    cache.close()
    del kv, kv3
    release(torch)


@pytest.mark.parametrize("index", [None, "ring"])
def test_hbm_gather_and_scatter_full_size(index, monkeypatch):
    # The measured HBM launches: one gather of 2,000 random pages of the
    # 20,000-page Qwen3 cache into a slot-layout device buffer, one scatter of
    # that buffer into 2,000 other pages (the default grids), with the page
    # ids in the kernel arguments (the default) or through the index ring.
    # Every gathered slot is the oracle's store of its page, every scattered
    # page the oracle's load of that slot, and no other page changes.
    if index:
        monkeypatch.setenv("EA_HBM_INDEX", index)
    torch = need_gpu()
    sh = W.QWEN3
    L, P, piece = sh.num_layers, sh.num_pages, sh.piece_bytes
    kv = torch.empty(sh.cache_bytes, dtype=torch.uint8, device="cuda")
    W.fill_bf16_normal(kv, W.SEED_DATA + 3)
    kv3 = kv.view(L, P, piece)
    cache = api.Cache(kv, P, L, sh.page_tokens, sh.num_kv_heads, sh.head_dim, sh.elem_bytes)
    r = W.rng(W.SEED_IDS + 3)
    n = W.QWEN3_STORE_PAGES
    src = W.distinct(r, P, n)
    dst = W.distinct(r, P, n, exclude=src)
    slot = L * piece
    staging = torch.full((n * slot,), POISON, dtype=torch.uint8, device="cuda")
    before = kv.clone()
    cache.gather(src, staging)
    cache.scatter(staging, dst)
    torch.cuda.synchronize()
    want = oracle_slots(sh, pages_to_host(torch, kv3, src))
    assert_rows_equal(staging.view(n, slot).cpu().numpy(), want, "gathered slots")
    want_l = oracle_pages(sh, want)
    del want
    got_l = pages_to_host(torch, kv3, dst)
    assert_rows_equal(got_l.transpose(1, 0, 2), want_l.transpose(1, 0, 2), "scattered pages")
    del want_l, got_l
    changed = changed_pages(torch, kv3, before.view(L, P, piece))
    assert np.isin(changed, dst).all(), np.setdiff1d(changed, dst)[:8]
    cache.close()
    del kv, kv3, staging, before
    release(torch)


@pytest.mark.parametrize("sh", [W.LAYERED, W.LAYERED_TP8], ids=lambda sh: sh.name)
def test_layered_fp8_prefix_full_size(sh):
    # the 64k-token fp8 prefix, and the same on one TP8 rank (1 KV head)
    torch = need_gpu()
    L, P, piece = sh.num_layers, sh.num_pages, sh.piece_bytes
    kv = torch.empty(sh.cache_bytes, dtype=torch.uint8, device="cuda")
    W.fill_random_bytes(kv, W.SEED_DATA)
    sc = torch.empty(L * P * 8, dtype=torch.uint8, device="cuda")
    W.fill_random_bytes(sc, W.SEED_DATA + 1)
    kv3, sc3 = kv.view(L, P, piece), sc.view(L, P, 8)
    cache = api.Cache(kv, P, L, sh.page_tokens, sh.num_kv_heads, sh.head_dim, sh.elem_bytes,
                      scales=sc)
    n = W.LAYERED_PREFIX_PAGES
    slot_bytes = L * piece + 512
    tier = api.Tier(cache, n * slot_bytes)
    assert tier.capacity == n and tier.slot_bytes == slot_bytes
    r = W.rng(W.SEED_IDS)
    src = W.distinct(r, P, n)
    dst = np.setdiff1d(np.arange(P), src)
    r.shuffle(dst)
    toks = W.tokens(W.SEED_TOKENS, n * sh.page_tokens)
    keys, _ = api.hash_blocks(toks, np.array([0, len(toks)]), sh.page_tokens)
    cnt, slots = tier.alloc(keys)
    assert cnt == n
    tier.store(cache, src, slots)
    tier.unpin(slots)
    d = torch.as_tensor(dst, device="cuda")
    s_ = torch.as_tensor(src, device="cuda")
    kv3[:, d] = 0xA5
    sc3[:, d] = 0x5A
    torch.cuda.synchronize()
    before3, before_sc3 = kv3.clone(), sc3.clone()
    h, hslots = tier.lookup(keys)
    assert h == n
    copy_s, cons_s = torch.cuda.Stream(), torch.cuda.Stream()
    events = [torch.cuda.Event() for _ in range(L)]
    sums = torch.zeros((L, n), dtype=torch.int64, device="cuda")
    tier.load_layered(cache, hslots, dst, copy_s, events)
    snaps = []
    with torch.cuda.stream(cons_s):
        for l in range(L):
            cons_s.wait_event(events[l])
            snaps.append((kv3[l].index_select(0, d).clone(), sc3[l].index_select(0, d).clone()))
            cache.layer_checksum(l, dst, sums[l], stream=cons_s)  # the consumer stand-in
    torch.cuda.synchronize()
    tier.unpin(hslots)
    for l in range(L):
        assert torch.equal(snaps[l][0], kv3[l].index_select(0, s_)), l
        assert torch.equal(snaps[l][1], sc3[l].index_select(0, s_)), l
    assert torch.equal(kv3[:, d], kv3[:, s_]) and torch.equal(sc3[:, d], sc3[:, s_])
    # every slot is the oracle's store of its source page (with scales), and
    # every destination page the oracle's layer-by-layer load of that image
    host = tier.host_view()
    src_pages = pages_to_host(torch, kv3, src)
    src_sc = sc3[:, s_].cpu().numpy()
    want = oracle_slots(sh, src_pages, src_sc)
    assert_rows_equal(host[hslots], want, "stored slots")
    o = oshape_of(sh, num_pages=n)
    ocache = np.zeros((L, n, piece), np.uint8)
    osc = np.zeros((L, n, 8), np.uint8)
    for l in range(L):
        oracle.load_layer(o, want, ocache.reshape(-1), osc.reshape(-1), np.arange(n),
                          np.arange(n, dtype=np.int32), l)
    got = pages_to_host(torch, kv3, dst)
    assert_rows_equal(got.transpose(1, 0, 2), ocache.transpose(1, 0, 2), "loaded pages")
    assert np.array_equal(sc3[:, d].cpu().numpy(), osc)
    # the consumer's per-layer checksums, taken right after each event, equal
    # the oracle's checksums of its own load
    o_full = oshape_of(sh, num_pages=n)
    got_sums = sums.cpu().numpy().view(np.uint64)
    for l in range(L):
        want_l = oracle.layer_checksum(o_full, ocache.reshape(-1), osc.reshape(-1), l,
                                       np.arange(n, dtype=np.int32))
        assert np.array_equal(got_sums[l], want_l), l
    # only destination pages changed since the poison was written
    assert np.isin(changed_pages(torch, kv3, before3), dst).all()
    assert np.isin(changed_pages(torch, sc3, before_sc3), dst).all()
    tier.close()
    cache.close()
    del kv, sc, kv3, sc3, before3, before_sc3
    release(torch)


def test_dense_scattered_calls_full_images():
    torch = need_gpu()
    sh = W.DENSE
    L, P, piece = sh.num_layers, sh.num_pages, sh.piece_bytes
    kv = torch.empty(sh.cache_bytes, dtype=torch.uint8, device="cuda")
    W.fill_bf16_normal(kv, W.SEED_DATA)
    cache = api.Cache(kv, P, L, sh.page_tokens, sh.num_kv_heads, sh.head_dim, sh.elem_bytes)
    tier = api.Tier(cache, W.DENSE_TIER_SLOTS * L * piece)
    host = tier.host_view()
    host[:] = 0
    torch.cuda.synchronize()
    o_cache = kv.cpu().numpy()
    o_tier = np.zeros_like(host)
    o = oshape_of(sh)
    drv = drivers.DenseScattered(cache, tier, sh)
    for i in range(W.DENSE_CALLS):
        op, pages, slots = drv.call(i)
        if op == "store":
            oracle.store_blocks(o, o_cache, None, o_tier, pages, slots)
        else:
            oracle.load_blocks(o, o_tier, o_cache, None, slots, pages)
    torch.cuda.synchronize()
    assert tier.stats()["evictions_total"] > 0  # the tier filled and recycled slots
    assert np.array_equal(host, o_tier)
    assert np.array_equal(kv.cpu().numpy(), o_cache)
    tier.close()
    cache.close()
    del kv
    release(torch)


def test_agent_pool_overlapped_streams():
    # loads and stores on two streams, a turn not waiting for the previous
    # store: metadata still equals the oracle's every turn, and every loaded
    # page still carries its key's pattern
    torch = need_gpu()
    sh = W.QWEN3
    kv = torch.empty(sh.cache_bytes, dtype=torch.uint8, device="cuda")
    cache = api.Cache(kv, sh.num_pages, sh.num_layers, sh.page_tokens, sh.num_kv_heads,
                      sh.head_dim, sh.elem_bytes)
    tier = api.Tier(cache, 16 << 30)  # 10,922 slots: the tier evicts early
    beta = sh.num_layers * sh.piece_bytes // sh.page_tokens
    kw = dict(kappa=256, block_tokens=sh.page_tokens, activity_window=16)
    pol = api.make_policy(beta_rank=beta, **kw)
    opol = oracle.make_policy(beta=beta, **kw)
    ot = oracle.Tier(oshape_of(sh), 16 << 30)
    pool = drivers.AgentPool(torch, cache, tier, kv, sh, pol, agents=16,
                             load_stream=torch.cuda.Stream(), store_stream=torch.cuda.Stream())
    hits = 0
    for t in range(4 * 16):
        rec = pool.turn()
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
        hits += h
    torch.cuda.synchronize()
    a, b = tier.export(), ot.export()
    for k in ("state", "pins", "keys", "lru"):
        assert np.array_equal(a[k], b[k]), k
    assert hits > 0 and tier.stats()["evictions_total"] > 0
    tier.close()
    cache.close()
    del kv
    release(torch)



def test_agent_pool_in_1024_token_chunks():
    # the paper's deployment parameters on one TP8 rank: 24 KiB per token,
    # 1,024-token host chunks (64 pages, 24 MiB), a 5 GiB tier (213 chunks),
    # 16 agents, kappa = 8 chunks; metadata equals the oracle's every turn
    torch = need_gpu()
    sh, C = W.QWEN3_TP8, W.CHUNK_PAGES
    kv = torch.empty(sh.cache_bytes, dtype=torch.uint8, device="cuda")
    cache = api.Cache(kv, sh.num_pages, sh.num_layers, sh.page_tokens, sh.num_kv_heads,
                      sh.head_dim, sh.elem_bytes)
    tier = api.Tier(cache, 5 << 30, chunk_pages=C)
    assert tier.capacity == 213
    beta = sh.num_layers * sh.piece_bytes // sh.page_tokens
    kw = dict(kappa=8, block_tokens=C * sh.page_tokens, activity_window=16)
    pol = api.make_policy(beta_rank=beta, **kw)
    opol = oracle.make_policy(beta=beta, **kw)
    oshape = oracle.make_shape(sh.num_pages, sh.num_layers, sh.page_tokens, sh.num_kv_heads,
                               sh.head_dim, sh.elem_bytes, chunk_pages=C)
    ot = oracle.Tier(oshape, 5 << 30)
    pool = drivers.AgentPool(torch, cache, tier, kv, sh, pol, agents=16)
    hits = declined = 0
    for t in range(4 * 16):
        rec = pool.turn()
        assert rec.loaded_ok, f"turn {t}: a loaded page differs from its chunk key's pattern"
        assert len(rec.keys) == rec.n_tokens // (C * sh.page_tokens)
        h, hs = ot.lookup(rec.keys)
        assert h == rec.hit and np.array_equal(hs, rec.hit_slots), t
        save, mask = ot.admission(opol, rec.n_tokens, rec.hit * C * sh.page_tokens, rec.agent,
                                  t, rec.keys)
        assert save == rec.save and np.array_equal(mask, rec.mask), t
        _, slots = ot.alloc(rec.keys, mask)
        assert np.array_equal(slots, rec.alloc_slots), t
        ok = slots >= 0
        ot.mark_stored(slots[ok])
        if ok.any():
            ot.unpin(slots[ok])
        if h:
            ot.unpin(hs)
        hits += h
        declined += int(not save)
    a, b = tier.export(), ot.export()
    for k in ("state", "pins", "keys", "lru"):
        assert np.array_equal(a[k], b[k]), k
    assert hits > 0 and tier.stats()["evictions_total"] > 0
    tier.close()
    cache.close()
    del kv
    release(torch)


def test_longest_prefix_on_one_tp8_rank():
    # a 262,144-token prefix (the serving configuration's maximum context),
    # 16,384 pages of one TP8 rank's share (384 KiB each, 6 GiB), stored to
    # shuffled slots and loaded back into other pages: every slot and every
    # loaded page against the oracle, no other page changed
    torch = need_gpu()
    sh = W.Shape("tp8_shard_long", 48, 1, 128, 2, 16, 2 * 16384 + 64)
    L, P, piece = sh.num_layers, sh.num_pages, sh.piece_bytes
    n = 16384
    kv = torch.empty(sh.cache_bytes, dtype=torch.uint8, device="cuda")
    W.fill_bf16_normal(kv, W.SEED_DATA)
    kv3 = kv.view(L, P, piece)
    cache = api.Cache(kv, P, L, sh.page_tokens, sh.num_kv_heads, sh.head_dim, sh.elem_bytes)
    tier = api.Tier(cache, n * L * piece)
    assert tier.capacity == n
    r = W.rng(131)
    src = W.distinct(r, P, n)
    dst = W.distinct(r, P, n, exclude=src)
    slots = r.permutation(n).astype(np.int64)
    before = kv.clone()
    tier.store(cache, src, slots)
    tier.load(cache, slots, dst)
    torch.cuda.synchronize()
    host = tier.host_view()
    want = oracle_slots(sh, pages_to_host(torch, kv3, src))
    assert_rows_equal(host[slots], want, "stored slots")
    want_l = oracle_pages(sh, want)
    del want
    got = pages_to_host(torch, kv3, dst)
    assert_rows_equal(got.transpose(1, 0, 2), want_l.transpose(1, 0, 2), "loaded pages")
    del want_l, got
    assert np.isin(changed_pages(torch, kv3, before.view(L, P, piece)), dst).all()
    tier.close()
    cache.close()
    del kv, kv3, before
    release(torch)
