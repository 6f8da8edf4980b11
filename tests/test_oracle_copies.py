"""Pins of the oracle's store and load (byte copies, so the result is unique):
numpy fancy-indexing restatements on tiny caches, round-trip identity,
untouched bytes, fp8 bit patterns (NaN encodings) and error paths."""
import numpy as np
import pytest

import oracle


def _setup(seed, P=24, L=3, T=4, H=2, D=8, s=2, scales=False, S=16):
    sh = oracle.make_shape(P, L, T, H, D, s, scales)
    sz = oracle.sizes(sh)
    rng = np.random.default_rng(seed)
    cache = rng.integers(0, 256, size=sz["cache"], dtype=np.uint8)
    sc = rng.integers(0, 256, size=sz["scales"], dtype=np.uint8) if scales else None
    tier = rng.integers(0, 256, size=(S, sz["slot"]), dtype=np.uint8)
    return sh, sz, rng, cache, sc, tier


def _np_store(sh, sz, cache, sc, tier, ids, slots):
    L, P = sh.num_layers, sh.num_pages
    c = cache.reshape(L, P, sz["piece"])
    out = tier.copy()
    for p, s in zip(ids, slots):
        out[s, :sz["page"]] = c[:, p, :].reshape(-1)
        if sc is not None:
            out[s, sz["page"]:sz["page"] + 8 * L] = sc.reshape(L, P, 8)[:, p, :].reshape(-1)
            out[s, sz["page"] + 8 * L:] = 0
    return out


@pytest.mark.parametrize("scales", [False, True])
def test_store_matches_numpy_restatement(scales):
    sh, sz, rng, cache, sc, tier = _setup(1, scales=scales)
    ids = rng.choice(sh.num_pages, 10, replace=False).astype(np.int32)
    slots = rng.choice(tier.shape[0], 10, replace=False).astype(np.int64)
    want = _np_store(sh, sz, cache, sc, tier, ids, slots)
    cache0 = cache.copy()
    oracle.store_blocks(sh, cache, sc, tier, ids, slots)
    assert np.array_equal(tier, want)
    assert np.array_equal(cache, cache0)  # the source pages are unchanged


def test_store_mask_skips_entries():
    sh, sz, rng, cache, sc, tier = _setup(2)
    ids = np.arange(6, dtype=np.int32)
    slots = np.array([0, 1, 1, 2, 3, 3])  # duplicates only among masked-out entries
    mask = np.array([1, 1, 0, 1, 1, 0], np.uint8)
    want = _np_store(sh, sz, cache, sc, tier, ids[mask == 1], slots[mask == 1])
    oracle.store_blocks(sh, cache, sc, tier, ids, slots, mask)
    assert np.array_equal(tier, want)


@pytest.mark.parametrize("scales", [False, True])
def test_round_trip_and_untouched_pages(scales):
    sh, sz, rng, cache, sc, tier = _setup(3, P=40, scales=scales, S=20)
    L, P = sh.num_layers, sh.num_pages
    src = rng.choice(P // 2, 12, replace=False).astype(np.int32)
    dst = (P // 2 + rng.choice(P // 2, 12, replace=False)).astype(np.int32)
    slots = rng.choice(tier.shape[0], 12, replace=False).astype(np.int64)
    oracle.store_blocks(sh, cache, sc, tier, src, slots)
    before = cache.copy()
    before_sc = None if sc is None else sc.copy()
    oracle.load_blocks(sh, tier, cache, sc, slots, dst)
    c = cache.reshape(L, P, -1)
    b = before.reshape(L, P, -1)
    assert np.array_equal(c[:, dst], b[:, src])  # round trip identity
    untouched = np.setdiff1d(np.arange(P), dst)
    assert np.array_equal(c[:, untouched], b[:, untouched])
    if sc is not None:
        s3, b3 = sc.reshape(L, P, 8), before_sc.reshape(L, P, 8)
        assert np.array_equal(s3[:, dst], b3[:, src])
        assert np.array_equal(s3[:, untouched], b3[:, untouched])


def test_load_per_layer_composes_to_full_load():
    sh, sz, rng, cache, sc, tier = _setup(4, scales=True)
    slots = rng.choice(tier.shape[0], 8, replace=False).astype(np.int64)
    dst = rng.choice(sh.num_pages, 8, replace=False).astype(np.int32)
    full, full_sc = cache.copy(), sc.copy()
    oracle.load_blocks(sh, tier, full, full_sc, slots, dst)
    lay, lay_sc = cache.copy(), sc.copy()
    L, P = sh.num_layers, sh.num_pages
    for l in range(L):
        oracle.load_layer(sh, tier, lay, lay_sc, slots, dst, l)
        # after layer l, layers 0..l of every destination already hold final bytes
        assert np.array_equal(lay.reshape(L, P, -1)[:l + 1], full.reshape(L, P, -1)[:l + 1])
    assert np.array_equal(lay, full) and np.array_equal(lay_sc, full_sc)


def test_fp8_nan_patterns_survive():
    sh = oracle.make_shape(4, 2, 16, 1, 16, 1, True)
    sz = oracle.sizes(sh)
    cache = np.tile(np.array([0x7F, 0xFF, 0x80, 0x00, 0x7E, 0xFE], np.uint8),
                    sz["cache"] // 6 + 1)[:sz["cache"]].copy()
    sc = np.frombuffer(np.array([np.nan, -np.inf, np.inf, -0.0], np.float32).tobytes() * (sz["scales"] // 16),
                       np.uint8).copy()
    tier = np.zeros((4, sz["slot"]), np.uint8)
    oracle.store_blocks(sh, cache, sc, tier, np.array([1, 3], np.int32), np.array([2, 0]))
    out = np.zeros_like(cache)
    out_sc = np.zeros_like(sc)
    oracle.load_blocks(sh, tier, out, out_sc, np.array([2, 0]), np.array([1, 3], np.int32))
    c, o = cache.reshape(2, 4, -1), out.reshape(2, 4, -1)
    assert np.array_equal(o[:, [1, 3]], c[:, [1, 3]])
    assert np.array_equal(out_sc.reshape(2, 4, 8)[:, [1, 3]], sc.reshape(2, 4, 8)[:, [1, 3]])


def test_trailer_padding_is_zeroed_in_stored_slots_only():
    sh, sz, rng, cache, sc, tier = _setup(5, scales=True)
    pad = slice(sz["page"] + 8 * sh.num_layers, sz["slot"])
    assert sz["slot"] - pad.start > 0
    before = tier.copy()
    oracle.store_blocks(sh, cache, sc, tier, np.array([0, 1], np.int32), np.array([0, 1]))
    assert not tier[:2, pad].any()
    assert np.array_equal(tier[2:], before[2:])


@pytest.mark.parametrize("bad", ["id_high", "id_neg", "slot_high", "dup_slot"])
def test_store_errors_write_nothing(bad):
    sh, sz, rng, cache, sc, tier = _setup(6)
    ids = np.array([0, 1, 2], np.int32)
    slots = np.array([0, 1, 2], np.int64)
    if bad == "id_high": ids[2] = sh.num_pages
    if bad == "id_neg": ids[1] = -1
    if bad == "slot_high": slots[2] = tier.shape[0]
    if bad == "dup_slot": slots[2] = 0
    before = tier.copy()
    with pytest.raises(oracle.OracleError) as e:
        oracle.store_blocks(sh, cache, sc, tier, ids, slots)
    assert e.value.code == oracle.EAO_EINVAL
    assert np.array_equal(tier, before)


@pytest.mark.parametrize("bad", ["dst_high", "slot_neg", "dup_dst", "scales_missing"])
def test_load_errors_write_nothing(bad):
    sh, sz, rng, cache, sc, tier = _setup(7, scales=(bad != "scales_missing"))
    if bad == "scales_missing":
        sh.has_scales = 1
    slots = np.array([0, 0, 1], np.int64)  # duplicate sources are allowed
    dst = np.array([3, 4, 5], np.int32)
    if bad == "dst_high": dst[0] = sh.num_pages
    if bad == "slot_neg": slots[0] = -1
    if bad == "dup_dst": dst[2] = 3
    before = cache.copy()
    with pytest.raises(oracle.OracleError):
        oracle.load_blocks(sh, tier, cache, sc, slots, dst)
    assert np.array_equal(cache, before)


def test_duplicate_sources_allowed():
    sh, sz, rng, cache, sc, tier = _setup(8)
    oracle.load_blocks(sh, tier, cache, sc, np.array([5, 5]), np.array([0, 1], np.int32))
    c = cache.reshape(sh.num_layers, sh.num_pages, -1)
    assert np.array_equal(c[:, 0], c[:, 1])


# ------------------------------------------------- chunked host slots (C > 1)

def _setup_chunked(seed, C, P=48, L=3, scales=False, S=6):
    sh = oracle.make_shape(P, L, 4, 2, 8, 2, scales, chunk_pages=C)
    sz = oracle.sizes(sh)
    rng = np.random.default_rng(seed)
    cache = rng.integers(0, 256, size=sz["cache"], dtype=np.uint8)
    sc = rng.integers(0, 256, size=sz["scales"], dtype=np.uint8) if scales else None
    tier = rng.integers(0, 256, size=(S, sz["slot"]), dtype=np.uint8)
    return sh, sz, rng, cache, sc, tier


def test_chunked_sizes():
    sh = oracle.make_shape(48, 3, 4, 2, 8, 2, True, chunk_pages=5)
    sz = oracle.sizes(sh)
    assert sz["piece"] == 2 * 4 * 2 * 8 * 2 and sz["page"] == 3 * sz["piece"]
    assert sz["payload"] == 5 * sz["page"]
    assert sz["trailer"] == 256  # 3 layers x 5 pages x 8 B = 120, padded
    assert sz["slot"] == sz["payload"] + 256
    # the paper's host chunk: 1,024 tokens = 64 pages of 16, 24 KiB/token/rank
    tp8 = oracle.sizes(oracle.make_shape(64, 48, 16, 1, 128, 2, chunk_pages=64))
    assert tp8["slot"] == 24 << 20
    # with fp32 scales: 48 layers x 64 pages x 8 B = 24,576 B, already a
    # multiple of 256
    fp8 = oracle.sizes(oracle.make_shape(64, 48, 16, 1, 128, 1, True, chunk_pages=64))
    assert fp8["trailer"] == 24576 and fp8["slot"] == (12 << 20) + 24576


@pytest.mark.parametrize("C,scales", [(2, False), (5, True), (8, True)])
def test_chunked_store_and_load_match_numpy_layout(C, scales):
    # slot layout [L][C][piece], trailer [L][C][2] float32 then zeros
    sh, sz, rng, cache, sc, tier = _setup_chunked(10 + C, C, scales=scales)
    L, P, piece = sh.num_layers, sh.num_pages, sz["piece"]
    n = 4
    ids = rng.choice(P, n * C, replace=True).astype(np.int32)  # repeats allowed
    slots = rng.choice(tier.shape[0], n, replace=False).astype(np.int64)
    want = tier.copy()
    c3 = cache.reshape(L, P, piece)
    for i in range(n):
        pages = ids[i * C:(i + 1) * C]
        want[slots[i], :sz["payload"]] = c3[:, pages, :].reshape(-1)  # [L][C][piece]
        if scales:
            s3 = sc.reshape(L, P, 8)
            want[slots[i], sz["payload"]:sz["payload"] + 8 * L * C] = s3[:, pages, :].reshape(-1)
            want[slots[i], sz["payload"] + 8 * L * C:] = 0
    oracle.store_blocks(sh, cache, sc, tier, ids, slots)
    assert np.array_equal(tier, want)
    # load the chunks back into distinct pages: chunk position c -> dst[i*C+c]
    dst = rng.choice(P, n * C, replace=False).astype(np.int32)
    before = cache.copy()
    before_sc = None if sc is None else sc.copy()
    oracle.load_blocks(sh, tier, cache, sc, slots, dst)
    got, was = cache.reshape(L, P, piece), before.reshape(L, P, piece)
    assert np.array_equal(got[:, dst], was[:, ids])
    rest = np.setdiff1d(np.arange(P), dst)
    assert np.array_equal(got[:, rest], was[:, rest])
    if scales:
        assert np.array_equal(sc.reshape(L, P, 8)[:, dst], before_sc.reshape(L, P, 8)[:, ids])
    # per-layer loads compose to the same image
    cache2 = before.copy()
    sc2 = None if sc is None else before_sc.copy()
    for layer in range(L):
        oracle.load_layer(sh, tier, cache2, sc2, slots, dst, layer)
    assert np.array_equal(cache2, cache)
    if scales:
        assert np.array_equal(sc2, sc)


def test_chunked_errors_write_nothing():
    sh, sz, rng, cache, sc, tier = _setup_chunked(30, 4)
    t0, c0 = tier.copy(), cache.copy()
    with pytest.raises(ValueError):  # not chunk_pages ids per slot
        oracle.store_blocks(sh, cache, sc, tier, np.arange(7, dtype=np.int32), [0, 1])
    with pytest.raises(oracle.OracleError):  # a page id out of range in the last chunk
        oracle.store_blocks(sh, cache, sc, tier, np.array([0, 1, 2, 3, 4, 5, 6, 48]), [0, 1])
    with pytest.raises(oracle.OracleError):  # duplicate destination across chunks
        oracle.load_blocks(sh, tier, cache, sc, [0, 1], np.array([0, 1, 2, 3, 4, 5, 6, 3]))
    assert np.array_equal(tier, t0) and np.array_equal(cache, c0)
    bad = oracle.make_shape(48, 3, 4, 2, 8, 2, chunk_pages=0)
    with pytest.raises(oracle.OracleError):
        oracle.store_blocks(bad, cache, None, tier, np.zeros(0, np.int32), np.zeros(0, np.int64))
