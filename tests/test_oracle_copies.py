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
