"""Pins of the oracle's LRU reference model (App. "Reference model",
Lemma 1, Proposition 1; section 3.2, Eq. 4 and Eq. 5).

The oracle simulates the tier one reference at a time.  These tests check it
against facts fixed independently of that simulation: reuse distances
counted by brute force over the stream (Eq. 4 / Lemma 1), the proposition's
containment of hits, the closed form of a backlogged round-robin pool,
Mattson's inclusion property, and the unbounded tier.
"""
import numpy as np
import pytest

import oracle


def keys_from_ids(ids, seed=7):
    """Distinct random 32-byte keys, one per distinct id."""
    ids = np.asarray(ids)
    r = np.random.default_rng(seed)
    table = r.integers(0, 256, size=(int(ids.max()) + 1 if len(ids) else 1, 32), dtype=np.uint8)
    return table[ids] if len(ids) else np.zeros((0, 32), np.uint8)


def previous_ref(ids):
    last, prev = {}, []
    for i, x in enumerate(ids):
        prev.append(last.get(x, -1))
        last[x] = i
    return prev


def brute_distance(ids, s, t):
    """Distinct chunks other than ids[t] referenced strictly between s and t."""
    return len(set(ids[s + 1:t]) - {ids[t]})


def random_ids(seed, n=160, pool=11):
    return np.random.default_rng(seed).integers(0, pool, size=n)


@pytest.mark.parametrize("seed", range(6))
def test_full_admission_hits_iff_distance_below_capacity(seed):
    ids = random_ids(seed)
    keys = keys_from_ids(ids)
    prev = previous_ref(ids)
    for K in range(0, 13):
        hits = oracle.lru_reference(keys, K)
        for t, s in enumerate(prev):
            want = s >= 0 and brute_distance(ids, s, t) < K
            assert bool(hits[t]) == want, (seed, K, t)


@pytest.mark.parametrize("seed", range(6))
def test_lemma1_with_declined_misses(seed):
    r = np.random.default_rng(100 + seed)
    ids = random_ids(100 + seed, n=200, pool=9)
    keys = keys_from_ids(ids)
    declined = r.random(len(ids)) < 0.35
    prev = previous_ref(ids)
    for K in (1, 3, 5, 8):
        hits = oracle.lru_reference(keys, K, declined)
        promoted = hits.astype(bool) | ~declined
        for t, s in enumerate(prev):
            if s < 0:
                assert not hits[t]
                continue
            p = len({ids[i] for i in range(s + 1, t) if promoted[i]} - {ids[t]})
            assert bool(hits[t]) == (bool(promoted[s]) and p < K), (seed, K, t)


def agent_like_ids(seed, agents=5, turns=6, start=6, grow=(1, 4), keep=0.8):
    """Round-robin agents whose chunk lists keep a leading share of the
    previous prompt and append fresh chunks (ids only, no keys)."""
    r = np.random.default_rng(seed)
    nxt = 0
    ctx = []
    for _ in range(agents):
        ctx.append(list(range(nxt, nxt + start)))
        nxt += start
    out, req = [], [0]
    for _ in range(turns):
        for a in range(agents):
            c = ctx[a]
            k = int(np.floor(keep * len(c)))
            n = len(c) + int(r.integers(grow[0], grow[1] + 1))
            c = c[:k] + list(range(nxt, nxt + n - k))
            nxt += n - k
            ctx[a] = c
            out.extend(c)
            req.append(len(out))
    return np.array(out), np.array(req)


@pytest.mark.parametrize("seed", range(4))
def test_proposition1_declines_never_lose_a_hit(seed):
    ids, _ = agent_like_ids(seed)
    keys = keys_from_ids(ids)
    n = len(ids)
    nxt = [-1] * n
    last = {}
    for i in range(n - 1, -1, -1):
        nxt[i] = last.get(ids[i], -1)
        last[ids[i]] = i
    for K in (10, 25, 40, 60, 80, 100, 130):
        full = oracle.lru_reference(keys, K).astype(bool)
        far = np.array([nxt[i] < 0 or brute_distance(ids, i, nxt[i]) >= K for i in range(n)])
        restricted = oracle.lru_reference(keys, K, far).astype(bool)
        assert np.all(restricted[full]), (seed, K)       # every hit survives
        assert restricted.sum() >= full.sum()


def test_declining_a_near_reuse_can_lose_a_hit():
    # a, b, a with K = 2: the second a is at distance 1 < 2 and hits; declining
    # the first a (next reuse at distance 1, inside capacity) loses that hit,
    # so the proposition's condition is needed
    keys = keys_from_ids([0, 1, 0])
    assert list(oracle.lru_reference(keys, 2)) == [0, 0, 1]
    assert list(oracle.lru_reference(keys, 2, [1, 0, 0])) == [0, 0, 0]


@pytest.mark.parametrize("A,n", [(4, 5), (8, 3), (2, 17)])
def test_round_robin_pool_survives_iff_tier_holds_every_context(A, n):
    # A agents, fixed contexts of n chunks, served round-robin: every chunk
    # is reused after the other A-1 contexts and the rest of its own, so
    # D = A*n - 1 and a returning request hits everything iff K >= A*n (the
    # working-set scale of Eq. 5, counted in chunks) and nothing otherwise
    ids = np.concatenate([np.arange(a * n, (a + 1) * n) for _ in range(3) for a in range(A)])
    keys = keys_from_ids(ids)
    for K in (0, n, A * n - 1, A * n, A * n + 7):
        hits = oracle.lru_reference(keys, K)
        assert not hits[:A * n].any()
        assert bool(hits[A * n:].all()) == (K >= A * n)
        assert bool(hits[A * n:].any()) == (K >= A * n)


@pytest.mark.parametrize("seed", range(5))
def test_inclusion_property(seed):
    ids, _ = agent_like_ids(50 + seed, agents=4, turns=5)
    keys = keys_from_ids(ids)
    prevh = oracle.lru_reference(keys, 0)
    for K in range(1, 70):
        h = oracle.lru_reference(keys, K)
        assert np.all(h >= prevh), K
        prevh = h


def test_unbounded_tier_hits_every_repeat():
    ids = random_ids(9, n=300, pool=40)
    keys = keys_from_ids(ids)
    seen, want = set(), []
    for x in ids:
        want.append(x in seen)
        seen.add(x)
    for K in (40, 41, 1000):
        assert list(oracle.lru_reference(keys, K).astype(bool)) == want


def test_edge_cases():
    empty = np.zeros((0, 32), np.uint8)
    assert len(oracle.lru_reference(empty, 5)) == 0
    keys = keys_from_ids([3, 3, 3])
    assert list(oracle.lru_reference(keys, 0)) == [0, 0, 0]
    assert list(oracle.lru_reference(keys, 1)) == [0, 1, 1]
    assert list(oracle.lru_reference(keys, 1, [1, 1, 1])) == [0, 0, 0]
    with pytest.raises(oracle.OracleError):
        oracle.lru_reference(keys, -1)


# ------------------------------------------- the host tier's own order

def tier_replay(keys, offs, K, save_flags):
    """Replay a stream on the oracle's host tier (lookup, deduplicated
    admission mask, allocation, store, unpin) and return the lookup hits
    per request.  Misses of requests with save_flags[j] == 0 are declined."""
    shape = oracle.make_shape(8, 1, 16, 1, 16, 2)  # 1 KiB slots
    slot = oracle.sizes(shape)["slot"]
    t = oracle.Tier(shape, K * slot)
    assert t.capacity == K
    pol = oracle.make_policy(kappa=1, block_tokens=16, beta=64, mode=oracle.ADMIT_ALWAYS)
    hits = []
    for j in range(len(offs) - 1):
        k = keys[offs[j]:offs[j + 1]]
        h, hs = t.lookup(k)
        save, mask = t.admission(pol, 16 * len(k), 16 * h, j, j, k)
        assert save == 1
        mask = mask & np.uint8(save_flags[j])
        _, slots = t.alloc(k, mask)
        ok = slots >= 0
        t.mark_stored(slots[ok])
        t.unpin(slots[ok])
        if h:
            t.unpin(hs)
        hits.append(h)
    t.close()
    return np.array(hits)


@pytest.mark.parametrize("seed", range(6))
def test_prefix_model_is_the_tier_order(seed):
    ids, offs = agent_like_ids(200 + seed, agents=6, turns=7, start=5, grow=(1, 5), keep=0.75)
    keys = keys_from_ids(ids, seed=200 + seed)
    r = np.random.default_rng(300 + seed)
    save = (r.random(len(offs) - 1) < [1.0, 0.8, 0.5, 0.8, 0.3, 0.0][seed]).astype(np.uint8)
    for K in (3, 12, 30, 55, 90, 400):
        want = tier_replay(keys, offs, K, save)
        got = oracle.lru_prefix_model(keys, offs, K, 1 - save)
        assert np.array_equal(got, want), (seed, K)


def test_prefix_model_edge_cases():
    keys = keys_from_ids([0, 1, 2, 0, 1, 2, 0, 9])
    offs = np.array([0, 3, 3, 6, 8])
    # unbounded tier: every repeated leading chunk hits
    assert list(oracle.lru_prefix_model(keys, offs, 100)) == [0, 0, 3, 1]
    # nothing admitted: nothing ever hits
    assert list(oracle.lru_prefix_model(keys, offs, 100, [1, 1, 1, 1])) == [0, 0, 0, 0]
    assert list(oracle.lru_prefix_model(keys, offs, 0)) == [0, 0, 0, 0]
    # K = 1: the request's own inserts are pinned, so only its first new chunk
    # fits and later ones are not inserted
    assert list(oracle.lru_prefix_model(keys, offs, 1)) == [0, 0, 1, 1]
    assert len(oracle.lru_prefix_model(np.zeros((0, 32), np.uint8), [0], 4)) == 0
    with pytest.raises(oracle.OracleError):
        oracle.lru_prefix_model(keys, [0, 5, 3], 4)
