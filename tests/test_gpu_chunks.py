"""GPU parity of host tiers with chunked slots (chunk_pages = C > 1: one key,
one LRU entry and one slot per C pages, the paper's 1,024-token host chunk;
Table "Serving configuration"), against the oracle byte for byte: both
transfer plans, inline and ring index paths, scales, masks, the layered
load, errors, and the TP8-shard shape at full size (24 MiB chunks)."""
import os

import numpy as np
import pytest

import oracle
from paper_2609_33762_amd import api, drivers, _native as N, workloads as W

from gpu_common import Pair, need_gpu

pytestmark = pytest.mark.gpu

PLANS = {"direct": N.EA_PLAN_DIRECT, "staged": N.EA_PLAN_STAGED}


def chunk_pair(C, slots, scales=False, seed=0):
    os.environ["EA_STAGING_MB"] = "1"  # several staging halves per call
    try:
        return Pair(256, 2, 16, 2, 64, 1 if scales else 2, slots, scales=scales, seed=seed,
                    chunk_pages=C)
    finally:
        os.environ.pop("EA_STAGING_MB")


@pytest.mark.parametrize("plan", list(PLANS))
@pytest.mark.parametrize("C,n,scales", [(4, 1, False), (4, 8, True), (4, 9, False),
                                         (4, 30, True), (16, 5, True), (64, 2, False)])
def test_chunked_store_and_load(plan, C, n, scales, monkeypatch, hbm_index=None):
    # n*C <= 32 page entries travel in kernel arguments; more go through the
    # index ring, except for the staged plan's HBM halves, whose page ids
    # travel in an argument block (through the ring with EA_HBM_INDEX=ring)
    if hbm_index:
        monkeypatch.setenv("EA_HBM_INDEX", hbm_index)
    p = chunk_pair(C, max(2 * n, 8), scales=scales, seed=100 + C + n)
    assert p.tier.chunk_pages == C and p.tier.slot_bytes == p.sizes["slot"]
    p.tier.set_plan(N.EA_DIR_BOTH, PLANS[plan])
    r = W.rng(200 + C * n)
    src = W.distinct(r, 256, n * C)
    dst = W.distinct(r, 256, n * C, exclude=src)
    slots = W.distinct(r, p.tier.capacity, n)
    p.tier.store(p.cache, src, slots)
    p.o_store(src, slots)
    p.assert_equal("store")
    p.tier.load(p.cache, slots, dst)
    p.o_load(slots, dst)
    p.assert_equal("load")
    p.close()


@pytest.mark.parametrize("C,n,scales", [(4, 30, True), (16, 5, True)])
def test_chunked_staged_halves_through_the_ring(C, n, scales, monkeypatch):
    # the staged plan with its HBM halves' page ids through the index ring
    test_chunked_store_and_load("staged", C, n, scales, monkeypatch, hbm_index="ring")


def test_chunked_mask_and_repeated_sources():
    p = chunk_pair(8, 12, scales=True, seed=7)
    r = W.rng(31)
    n = 10
    src = r.integers(0, 256, size=n * 8).astype(np.int32)  # sources may repeat
    slots = np.array([0, 1, 1, 2, 3, 3, 4, 5, 6, 6])  # repeats only where masked out
    mask = np.array([1, 1, 0, 1, 1, 0, 1, 1, 1, 0], np.uint8)
    p.tier.store(p.cache, src, slots, mask)
    p.o_store(src, slots, mask)
    p.assert_equal("masked store")
    p.close()


@pytest.mark.parametrize("C,n", [(4, 6), (8, 10)])
def test_chunked_layered_load(C, n):
    torch = need_gpu()
    p = chunk_pair(C, 2 * n, scales=True, seed=40 + C)
    r = W.rng(50 + C)
    src = W.distinct(r, 256, n * C)
    dst = W.distinct(r, 256, n * C, exclude=src)
    slots = W.distinct(r, p.tier.capacity, n)
    p.tier.store(p.cache, src, slots)
    p.o_store(src, slots)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    evs = [torch.cuda.Event() for _ in range(2)]
    p.tier.load_layered(p.cache, slots, dst, s, evs)
    for layer in range(2):
        oracle.load_layer(p.oshape, p.o_tier, p.o_cache, p.o_sc, slots, dst, layer)
    p.assert_equal("layered load")
    p.close()


def test_chunked_errors_move_nothing():
    torch = need_gpu()
    p = chunk_pair(4, 8, seed=9)
    r = W.rng(60)
    src = W.distinct(r, 256, 16)
    p.tier.store(p.cache, src, [0, 1, 2, 3])
    p.o_store(src, [0, 1, 2, 3])
    p.snapshot()
    with pytest.raises(ValueError):  # not C page ids per slot
        p.tier.load(p.cache, [0, 1], src[:7])
    lib = N.load()
    dup = np.array([10, 11, 12, 13, 14, 15, 16, 10], np.int32)  # repeated destination
    sl = np.array([0, 1], np.int64)
    s = torch.cuda.current_stream().cuda_stream
    assert lib.ea_load_blocks(p.tier._h, p.cache.handle, sl.ctypes.data, dup.ctypes.data, 2,
                              s) == N.EA_EINVAL
    bad = np.array([0, 1, 2, 3, 4, 5, 6, 256], np.int32)  # page out of range
    assert lib.ea_store_blocks(p.cache.handle, p.tier._h, bad.ctypes.data, sl.ctypes.data,
                               None, 2, s) == N.EA_EINVAL
    p.assert_equal("after rejected calls")
    p.close()


def test_tp8_shard_chunked_turn_full_size():
    # one rank of TP8 (24 KiB per token), 1,024-token chunks of 24 MiB:
    # refill 31 chunks (1,984 pages), restore a 23-chunk prefix (1,472 pages)
    torch = need_gpu()
    sh, C = W.QWEN3_TP8, W.CHUNK_PAGES
    L, P, piece = sh.num_layers, sh.num_pages, sh.piece_bytes
    kv = torch.empty(sh.cache_bytes, dtype=torch.uint8, device="cuda")
    W.fill_bf16_normal(kv, W.SEED_DATA)
    kv3 = kv.view(L, P, piece)
    cache = api.Cache(kv, P, L, sh.page_tokens, sh.num_kv_heads, sh.head_dim, sh.elem_bytes)
    tier = api.Tier(cache, 16 << 30, chunk_pages=C)
    assert tier.slot_bytes == 24 << 20 and tier.capacity == 682
    r = W.rng(W.SEED_IDS)
    n_l, n_s = 23, 31
    prefix = W.distinct(r, P, n_l * C)
    refill = W.distinct(r, P, n_s * C, exclude=prefix)
    dst = W.distinct(r, P, n_l * C, exclude=np.concatenate([prefix, refill]))
    toks = W.tokens(W.SEED_TOKENS, n_l * C * sh.page_tokens)
    pkeys, _ = api.hash_blocks(toks, np.array([0, len(toks)]), C * sh.page_tokens)
    assert len(pkeys) == n_l
    cnt, pslots = tier.alloc(pkeys)
    assert cnt == n_l
    tier.store(cache, prefix, pslots)
    tier.unpin(pslots)
    rkeys = W.rng(8).integers(0, 256, size=(n_s, 32), dtype=np.uint8)
    cnt, sslots = tier.alloc(rkeys)
    assert cnt == n_s
    s_store, s_load = torch.cuda.Stream(), torch.cuda.Stream()
    h, hslots = tier.lookup(pkeys)
    assert h == n_l
    tier.load(cache, hslots, dst, stream=s_load)
    tier.store(cache, refill, sslots, stream=s_store)
    torch.cuda.synchronize()
    tier.unpin(sslots)
    tier.unpin(hslots)
    # round trip of every page, and every written slot against the oracle
    assert torch.equal(kv3[:, torch.as_tensor(dst, device="cuda")],
                       kv3[:, torch.as_tensor(prefix, device="cuda")])
    host = tier.host_view()
    o = oracle.make_shape(n_s * C, L, sh.page_tokens, sh.num_kv_heads, sh.head_dim,
                          sh.elem_bytes, chunk_pages=C)
    mini = drivers.read_pages(torch, kv3, refill).cpu().numpy()
    mini_cache = np.ascontiguousarray(mini.reshape(n_s * C, L, piece).transpose(1, 0, 2))
    want = np.zeros((n_s, tier.slot_bytes), np.uint8)
    oracle.store_blocks(o, mini_cache.reshape(-1), None, want, np.arange(n_s * C),
                        np.arange(n_s))
    assert np.array_equal(host[sslots], want)
    tier.close()
    cache.close()
    del kv, kv3
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
