"""GPU parity of store / load / layered load / gather / scatter against the
oracle, byte for byte on the full cache and tier images of small caches
(several pieces per page, ragged batches, both transfer plans, fp8 with
scales, masks, error paths, cross-stream hazards)."""
import os

import numpy as np
import pytest

import oracle
from paper_2609_33762_amd import _native as N
from paper_2609_33762_amd import workloads as W

from gpu_common import Pair, need_gpu

pytestmark = pytest.mark.gpu

PLANS = {"direct": N.EA_PLAN_DIRECT, "staged": N.EA_PLAN_STAGED}


def tiny_pair(**kw):
    sh = W.TINY
    return Pair(sh.num_pages, sh.num_layers, sh.page_tokens, sh.num_kv_heads, sh.head_dim,
                sh.elem_bytes, kw.pop("slots", W.TINY_TIER_SLOTS), **kw)


@pytest.mark.parametrize("plan", list(PLANS))
def test_tiny_config_store_then_load(plan):
    # Tiny workload: 32 random pages stored, loaded into 32 other free pages
    p = tiny_pair(seed=11)
    p.tier.set_plan(N.EA_DIR_BOTH, PLANS[plan])
    r = W.rng(W.SEED_IDS)
    src = W.distinct(r, W.TINY.num_pages, 32)
    dst = W.distinct(r, W.TINY.num_pages, 32, exclude=src)
    slots = W.distinct(r, p.tier.capacity, 32)
    p.tier.store(p.cache, src, slots)
    p.o_store(src, slots)
    p.assert_equal("store")
    p.tier.load(p.cache, slots, dst)
    p.o_load(slots, dst)
    p.assert_equal("load")
    # round trip: the destination pages now hold the source pages
    kv = p.kv.cpu().numpy().reshape(W.TINY.num_layers, W.TINY.num_pages, -1)
    assert np.array_equal(kv[:, dst], kv[:, src])
    p.close()


@pytest.mark.parametrize("plan", list(PLANS))
@pytest.mark.parametrize("n", [1, 31, 32, 33, 100, 200])
def test_ragged_batches_and_masks(plan, n):
    # n <= 32 travels in kernel arguments, larger batches through index upload
    os.environ["EA_STAGING_MB"] = "1"  # 32 slots per staging half: several chunks
    try:
        p = tiny_pair(seed=20 + n, slots=256)
    finally:
        os.environ.pop("EA_STAGING_MB")
    p.tier.set_plan(N.EA_DIR_BOTH, PLANS[plan])
    r = W.rng(1000 + n)
    src = W.distinct(r, W.TINY.num_pages, n)
    slots = W.distinct(r, p.tier.capacity, n)
    if n > 40:  # a run of 40 consecutive slots for the DMA coalescing
        rest = W.distinct(r, p.tier.capacity, n - 40, exclude=np.arange(100, 140))
        slots = np.concatenate([np.arange(100, 140), rest])
    mask = (r.random(n) < 0.8).astype(np.uint8)
    mask[0] = 1
    p.tier.store(p.cache, src, slots, mask)
    p.o_store(src, slots, mask)
    p.assert_equal("masked store")
    keep = mask == 1
    dst = W.distinct(r, W.TINY.num_pages, int(keep.sum()))
    p.tier.load(p.cache, slots[keep], dst)
    p.o_load(slots[keep], dst)
    p.assert_equal("load")
    p.close()


@pytest.mark.parametrize("plan", list(PLANS))
def test_fp8_with_scales_and_duplicate_sources(plan):
    p = Pair(48, 3, 16, 2, 64, 1, 40, scales=True, seed=5)
    p.tier.set_plan(N.EA_DIR_BOTH, PLANS[plan])
    r = W.rng(7)
    src = W.distinct(r, 48, 36)
    slots = W.distinct(r, 40, 36)
    p.tier.store(p.cache, src, slots)
    p.o_store(src, slots)
    p.assert_equal("fp8 store")
    # the same slot may feed several destination pages
    lslots = np.concatenate([slots[:20], slots[:5]])
    dst = W.distinct(r, 48, 25)
    p.tier.load(p.cache, lslots, dst)
    p.o_load(lslots, dst)
    p.assert_equal("fp8 load")
    p.close()


def test_errors_move_nothing():
    p = tiny_pair(seed=3)
    before_tier = p.tier.host_view().copy()
    before = p.kv.cpu().numpy()
    cases = [
        ("store", dict(ids=[0, 1], slots=[0, 0])),               # duplicate destination slot
        ("store", dict(ids=[0, W.TINY.num_pages], slots=[0, 1])),
        ("store", dict(ids=[0, 1], slots=[0, p.tier.capacity])),
        ("load", dict(slots=[0, 1], dst=[5, 5])),                 # duplicate destination page
        ("load", dict(slots=[-1, 1], dst=[5, 6])),
        ("load", dict(slots=[0, 1], dst=[5, W.TINY.num_pages])),
    ]
    for op, a in cases:
        with pytest.raises(N.EAError) as e:
            if op == "store":
                p.tier.store(p.cache, a["ids"], a["slots"])
            else:
                p.tier.load(p.cache, a["slots"], a["dst"])
        assert e.value.code == N.EA_EINVAL
    p.torch.cuda.synchronize()
    assert np.array_equal(p.tier.host_view(), before_tier)
    assert np.array_equal(p.kv.cpu().numpy(), before)
    st = p.tier.stats()
    assert st["store_calls"] == 0 and st["load_calls"] == 0
    p.close()


def test_peak_probe_refuses_a_tier_in_use():
    # the probe overwrites the first slots; with one of them allocated it
    # must move nothing
    torch = need_gpu()
    p = tiny_pair(seed=4)
    slot = p.sizes["slot"]
    buf = torch.empty(4 * slot, dtype=torch.uint8, device="cuda")
    assert p.tier.peak_probe(buf, 2 * slot, N.EA_DIR_BOTH, 1) > 0  # empty tier: fine
    key = np.arange(32, dtype=np.uint8)[None, :]
    cnt, slots = p.tier.alloc(key)
    assert cnt == 1 and slots[0] == 0
    p.tier.store(p.cache, [7], slots)
    torch.cuda.synchronize()
    before = p.tier.host_view().copy()
    for direction in (N.EA_DIR_STORE, N.EA_DIR_LOAD, N.EA_DIR_BOTH):
        with pytest.raises(N.EAError) as e:
            p.tier.peak_probe(buf, slot, direction, 1)
        assert e.value.code == N.EA_EINVAL
    torch.cuda.synchronize()
    assert np.array_equal(p.tier.host_view(), before)
    p.tier.unpin(slots)
    p.close()


def test_load_on_another_stream_waits_for_the_store():
    torch = need_gpu()
    p = tiny_pair(seed=9, slots=256)
    r = W.rng(9)
    src = W.distinct(r, W.TINY.num_pages, 120)
    slots = W.distinct(r, p.tier.capacity, 120)
    dst = W.distinct(r, W.TINY.num_pages, 120, exclude=src)
    a, b = torch.cuda.Stream(), torch.cuda.Stream()
    # a long store on stream a, the load of the same slots on stream b at once
    p.tier.store(p.cache, src, slots, stream=a)
    p.tier.load(p.cache, slots, dst, stream=b)
    p.o_store(src, slots)
    p.o_load(slots, dst)
    p.assert_equal("cross-stream")
    p.close()


@pytest.mark.parametrize("n", [20, 300])
def test_layered_load_events_mark_finished_layers(n):
    torch = need_gpu()
    L, P = 6, 700
    p = Pair(P, L, 16, 2, 64, 1, 320, scales=True, seed=31)
    r = W.rng(31)
    src = W.distinct(r, P, n)
    slots = W.distinct(r, 320, n)
    p.tier.store(p.cache, src, slots)
    p.o_store(src, slots)
    dst = W.distinct(r, P, n, exclude=src)
    # poison the destination pages so a premature event would show
    kv3 = p.kv.view(L, P, -1)
    kv3[:, torch.as_tensor(dst, device="cuda")] = 0xA5
    p.snapshot()
    copy_s, cons_s = torch.cuda.Stream(), torch.cuda.Stream()
    events = [torch.cuda.Event() for _ in range(L)]
    p.tier.load_layered(p.cache, slots, dst, copy_s, events)
    snaps = []
    d = torch.as_tensor(dst, device="cuda")
    with torch.cuda.stream(cons_s):
        for l in range(L):
            cons_s.wait_event(events[l])
            snaps.append(kv3[l].index_select(0, d).clone())
    torch.cuda.synchronize()
    p.o_load(slots, dst)
    p.assert_equal("layered end state")
    want = p.o_cache.reshape(L, P, -1)
    for l in range(L):
        assert np.array_equal(snaps[l].cpu().numpy(), want[l][dst]), l
    p.close()


@pytest.mark.parametrize("index", [None, "ring"])
@pytest.mark.parametrize("n", [7, 150])
def test_gather_scatter_through_device_buffer(n, index, monkeypatch):
    # page ids in the kernel arguments (the default for 33-2,048 pages) or
    # through the mapped index ring
    if index:
        monkeypatch.setenv("EA_HBM_INDEX", index)
    torch = need_gpu()
    p = Pair(256, 4, 16, 2, 64, 2, 8, scales=True, seed=41)
    slot = p.sizes["slot"]
    r = W.rng(41)
    src = W.distinct(r, 256, n)
    dst = W.distinct(r, 256, n, exclude=src if n < 128 else None)
    buf = torch.full((n * slot,), 0x5A, dtype=torch.uint8, device="cuda")
    p.cache.gather(src, buf)
    # oracle: the gather buffer is a tier whose slot i holds entry i
    want = np.full((n, slot), 0x5A, np.uint8)
    oracle.store_blocks(p.oshape, p.o_cache, p.o_sc, want, src, np.arange(n))
    torch.cuda.synchronize()
    assert np.array_equal(buf.cpu().numpy().reshape(n, slot), want)
    p.cache.scatter(buf, dst)
    oracle.load_blocks(p.oshape, want, p.o_cache, p.o_sc, np.arange(n), dst)
    p.assert_equal("scatter")
    p.close()


@pytest.mark.parametrize("n", [2048, 2049])
def test_gather_scatter_at_the_argument_limit(n):
    # up to 2,048 page ids travel in the kernel arguments, one more goes
    # through the index ring: both sides of the limit, every gathered slot
    # and every page of the cache against the oracle
    torch = need_gpu()
    P = 4200
    p = Pair(P, 2, 16, 2, 64, 2, 8, scales=True, seed=47)
    slot = p.sizes["slot"]
    r = W.rng(47)
    src = W.distinct(r, P, n)
    dst = W.distinct(r, P, n, exclude=src)
    buf = torch.full((n * slot,), 0x5A, dtype=torch.uint8, device="cuda")
    p.cache.gather(src, buf)
    want = np.full((n, slot), 0x5A, np.uint8)
    oracle.store_blocks(p.oshape, p.o_cache, p.o_sc, want, src, np.arange(n))
    torch.cuda.synchronize()
    assert np.array_equal(buf.cpu().numpy().reshape(n, slot), want)
    p.cache.scatter(buf, dst)
    oracle.load_blocks(p.oshape, want, p.o_cache, p.o_sc, np.arange(n), dst)
    p.assert_equal("scatter")
    p.close()


def test_failed_tier_allocation_leaves_the_library_usable():
    # an absurd capacity (2^62 bytes, beyond any address space) fails with
    # EA_ENOMEM before anything is pinned; later launches still report their
    # own status and move the right bytes
    p = tiny_pair(seed=5)
    from paper_2609_33762_amd import api
    with pytest.raises(N.EAError) as e:
        api.Tier(p.cache, 1 << 62)
    assert e.value.code == N.EA_ENOMEM
    r = W.rng(5)
    src = W.distinct(r, W.TINY.num_pages, 40)
    dst = W.distinct(r, W.TINY.num_pages, 40, exclude=src)
    slots = W.distinct(r, p.tier.capacity, 40)
    p.tier.store(p.cache, src, slots)
    p.tier.load(p.cache, slots, dst)
    p.o_store(src, slots)
    p.o_load(slots, dst)
    p.assert_equal("after a failed tier allocation")
    p.close()


@pytest.mark.parametrize("placement", ["hardware", "index"])
@pytest.mark.parametrize("masks", [(0x1, 0x2), (0x80, 0x40), (0x3, 0xC), (0xFF, 0xFF),
                                   (0x11, 0x22), (0x7F, 0x1)])
def test_any_xcd_masks_copy_every_piece(masks, placement, monkeypatch):
    # Work goes only to workgroups on the XCDs of the store and load masks
    # (the XCD the hardware reports, or the workgroup index when the probe
    # fails or EA_XCD_PLACEMENT=index); whatever the masks and the placement,
    # every piece is copied exactly once.
    monkeypatch.setenv("EA_XCD_STORE", hex(masks[0]))
    monkeypatch.setenv("EA_XCD_LOAD", hex(masks[1]))
    if placement == "index":
        monkeypatch.setenv("EA_XCD_PLACEMENT", "index")
    p = tiny_pair(seed=40 + masks[0], slots=256)
    monkeypatch.delenv("EA_XCD_STORE")
    monkeypatch.delenv("EA_XCD_LOAD")
    monkeypatch.delenv("EA_XCD_PLACEMENT", raising=False)
    r = W.rng(masks[0] * 7 + masks[1])
    for n in (5, 120):  # kernel arguments, then the index ring
        src = W.distinct(r, W.TINY.num_pages, n)
        dst = W.distinct(r, W.TINY.num_pages, n, exclude=src)
        slots = W.distinct(r, p.tier.capacity, n)
        p.tier.store(p.cache, src, slots)
        p.tier.load(p.cache, slots, dst)
        p.o_store(src, slots)
        p.o_load(slots, dst)
        p.assert_equal(f"masks {masks} n={n}")
    p.close()


@pytest.mark.parametrize("hbm_index", [None, "ring"])
@pytest.mark.parametrize("placement", ["hardware", "index"])
def test_one_workgroup_runs_many_index_batches(placement, hbm_index, monkeypatch):
    # Kernels fetch page and slot indices 64 units per wave at a time.  With
    # one working workgroup (four waves) on one XCD, 600 pages of 4 layers
    # give each wave about 600 units: ten index batches, the last one
    # partial.  Store, load, layered load, gather and scatter (page ids in
    # the kernel arguments or through the index ring), full images against
    # the oracle.
    if hbm_index:
        monkeypatch.setenv("EA_HBM_INDEX", hbm_index)
    torch = need_gpu()
    for k, v in {"EA_LINK_WG": "1", "EA_LINK_WG_LAYERED": "1", "EA_XCD_STORE": "0x1",
                 "EA_XCD_LOAD": "0x1", "EA_GRID_GATHER": "1", "EA_GRID_SCATTER": "1",
                 "EA_GRID_HBM": "1"}.items():
        monkeypatch.setenv(k, v)
    if placement == "index":
        monkeypatch.setenv("EA_XCD_PLACEMENT", "index")
    L, P, S, n = 4, 2000, 640, 600
    p = Pair(P, L, 16, 1, 32, 2, S, scales=True, seed=61)  # 2 KiB pieces
    r = W.rng(61)
    src = W.distinct(r, P, n)
    dst = W.distinct(r, P, n, exclude=src)
    slots = W.distinct(r, S, n)
    p.tier.store(p.cache, src, slots)
    p.o_store(src, slots)
    p.assert_equal("store, one workgroup")
    p.tier.load(p.cache, slots, dst)
    p.o_load(slots, dst)
    p.assert_equal("load, one workgroup")
    dst2 = W.distinct(r, P, n, exclude=np.concatenate([src, dst]))
    copy_s = torch.cuda.Stream()
    events = [torch.cuda.Event() for _ in range(L)]
    p.tier.load_layered(p.cache, slots, dst2, copy_s, events)
    torch.cuda.synchronize()
    p.o_load(slots, dst2)
    p.assert_equal("layered load, one workgroup")
    slot = p.sizes["slot"]
    buf = torch.full((n * slot,), 0x5A, dtype=torch.uint8, device="cuda")
    p.cache.gather(src, buf)
    want = np.full((n, slot), 0x5A, np.uint8)
    oracle.store_blocks(p.oshape, p.o_cache, p.o_sc, want, src, np.arange(n))
    torch.cuda.synchronize()
    assert np.array_equal(buf.cpu().numpy().reshape(n, slot), want)
    dst3 = np.setdiff1d(np.arange(P), src)[:n]
    p.cache.scatter(buf, dst3)
    oracle.load_blocks(p.oshape, want, p.o_cache, p.o_sc, np.arange(n), dst3)
    p.assert_equal("scatter, one workgroup")
    p.close()


def test_device_buffer_sizes_are_checked():
    # gather / scatter buffers and layer events must match the call; a short
    # one is refused and nothing is launched
    torch = need_gpu()
    import ctypes as C
    p = tiny_pair(seed=62)
    slot = p.sizes["slot"]
    n = 10
    buf = torch.full((n * slot - 16,), 0x5A, dtype=torch.uint8, device="cuda")
    ids = np.arange(n, dtype=np.int32)
    with pytest.raises(ValueError):
        p.cache.gather(ids, buf)
    with pytest.raises(ValueError):
        p.cache.scatter(buf, ids)
    lib = N.load()
    assert lib.ea_gather_blocks(p.cache.handle, ids.ctypes.data, n, buf.data_ptr(),
                                buf.numel(), None) == N.EA_EINVAL
    assert lib.ea_scatter_blocks(p.cache.handle, buf.data_ptr(), buf.numel(), ids.ctypes.data,
                                 n, None) == N.EA_EINVAL
    torch.cuda.synchronize()
    assert (buf.cpu().numpy() == 0x5A).all()
    slots = np.arange(4, dtype=np.int64)
    p.tier.store(p.cache, ids[:4], slots)
    events = [torch.cuda.Event() for _ in range(W.TINY.num_layers - 1)]
    with pytest.raises(ValueError):
        p.tier.load_layered(p.cache, slots, ids[4:8], torch.cuda.Stream(), events)
    evs = (C.c_void_p * 1)()
    dst = ids[4:8].copy()
    assert lib.ea_load_blocks_layered(p.tier._h, p.cache.handle, slots.ctypes.data,
                                      dst.ctypes.data, 4, None, evs, 1) == N.EA_EINVAL
    p.close()


@pytest.mark.parametrize("scales", [False, True])
@pytest.mark.parametrize("n", [1, 37, 300])
def test_layer_checksum_matches_the_oracle(scales, n):
    # the consumer stand-in of the layered load, on random bytes (fp8 NaN
    # patterns included), ragged page lists with repeats
    torch = need_gpu()
    L, P = 3, 400
    p = Pair(P, L, 16, 2, 64, 1, 8, scales=scales, seed=70 + n)
    r = W.rng(70 + n)
    pages = r.integers(0, P, size=n).astype(np.int32)
    out = torch.full((n + 3,), 7, dtype=torch.int64, device="cuda")
    for layer in range(L):
        p.cache.layer_checksum(layer, pages, out)
        want = oracle.layer_checksum(p.oshape, p.o_cache, p.o_sc, layer, pages)
        torch.cuda.synchronize()
        got = out.cpu().numpy().view(np.uint64)
        assert np.array_equal(got[:n], want), layer
        assert (got[n:] == 7).all()
    p.close()
