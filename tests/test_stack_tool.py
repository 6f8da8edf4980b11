"""Reuse-distance capacity tool of libea (ea_reuse_distances,
ea_prefix_coverage; section 3.2 Eq. 4, App. "Prefix coverage from a
reference stream") against the oracle's LRU reference model.

Host-only calls: these run without a GPU.  A reference hits in an LRU tier of
K chunks that admits every miss exactly when 0 <= prev_dist < K, so the
distances are checked against the oracle's hits at every capacity that can
change the answer, and the coverage against the oracle's leading hits.
"""
import numpy as np
import pytest

import oracle
from paper_2609_33762_amd import _native as N
from paper_2609_33762_amd import api
from paper_2609_33762_amd import workloads as W
from paper_2609_33762_amd._native import EAError


def small_stream(seed, n=240, pool=14):
    r = np.random.default_rng(seed)
    table = r.integers(0, 256, size=(pool, 32), dtype=np.uint8)
    return table[r.integers(0, pool, size=n)]


@pytest.mark.parametrize("seed", range(5))
def test_distances_reproduce_oracle_hits_at_every_capacity(seed):
    refs = small_stream(seed)
    prev, nxt = api.reuse_distances(refs)
    assert prev.max() < 14
    for K in range(0, 16):
        want = oracle.lru_reference(refs, K).astype(bool)
        assert np.array_equal((prev >= 0) & (prev < K), want), K


@pytest.mark.parametrize("seed", range(3))
def test_next_distance_is_the_next_references_previous_distance(seed):
    refs = small_stream(10 + seed, n=500, pool=30)
    prev, nxt = api.reuse_distances(refs)
    ids = [bytes(k) for k in refs]
    later = {}
    for i in range(len(ids) - 1, -1, -1):
        t = later.get(ids[i], -1)
        assert nxt[i] == (prev[t] if t >= 0 else -1), i
        later[ids[i]] = i


@pytest.mark.parametrize("seed", range(3))
def test_coverage_matches_oracle_on_agent_stream(seed):
    keys, offs = W.chunk_stream(seed, agents=12, turns=8, start_chunks=32, max_chunks=256,
                                growth_chunks=(3, 20), keep=0.98)
    prev, _ = api.reuse_distances(keys)
    total = int(offs[-1])
    assert len(keys) == total
    # capacities around the pool's working set (about agents x mean context)
    caps = np.array([0, 1, 100, 400, 900, 1300, 1700, 2200, 3000, 10**9])
    cov = api.prefix_coverage(prev, offs, caps)
    for c, K in enumerate(caps):
        hits = oracle.lru_reference(keys, min(int(K), total + 1)).astype(bool)
        for j in range(len(offs) - 1):
            h = hits[offs[j]:offs[j + 1]]
            lead = int(np.argmin(h)) if not h.all() else len(h)
            assert cov[j, c] == lead, (K, j)
    # coverage never shrinks as the tier grows
    assert np.all(np.diff(cov, axis=1) >= 0)


def test_round_robin_closed_form():
    A, n = 6, 9
    table = np.random.default_rng(3).integers(0, 256, size=(A * n, 32), dtype=np.uint8)
    ids = np.concatenate([np.arange(a * n, (a + 1) * n) for _ in range(4) for a in range(A)])
    prev, nxt = api.reuse_distances(table[ids])
    assert np.all(prev[:A * n] == -1) and np.all(prev[A * n:] == A * n - 1)
    assert np.all(nxt[:-A * n] == A * n - 1) and np.all(nxt[-A * n:] == -1)
    offs = np.arange(0, len(ids) + 1, n)
    cov = api.prefix_coverage(prev, offs, [A * n - 1, A * n])
    assert np.all(cov[:A, :] == 0)
    assert np.all(cov[A:, 0] == 0) and np.all(cov[A:, 1] == n)


def test_empty_and_degenerate_inputs():
    prev, nxt = api.reuse_distances(np.zeros((0, 32), np.uint8))
    assert len(prev) == 0 and len(nxt) == 0
    one = np.full((1, 32), 7, np.uint8)
    assert list(api.reuse_distances(one)[0]) == [-1]
    same = np.full((4, 32), 9, np.uint8)
    prev, nxt = api.reuse_distances(same)
    assert list(prev) == [-1, 0, 0, 0] and list(nxt) == [0, 0, 0, -1]
    # empty requests and no capacities
    cov = api.prefix_coverage(prev, [0, 0, 2, 2, 4], [0, 1])
    assert cov.tolist() == [[0, 0], [0, 0], [0, 0], [0, 2]]
    assert api.prefix_coverage(prev, [0, 4], []).shape == (1, 0)
    assert api.prefix_coverage(prev, [0], [1, 2]).shape == (0, 2)


def test_argument_errors():
    lib = N.load()
    assert lib.ea_reuse_distances(None, 3, None, None) == -1
    assert lib.ea_reuse_distances(None, -1, None, None) == -1
    prev = np.zeros(4, np.int64)
    cov = np.zeros(8, np.int64)
    bad_offs = np.array([0, 3, 2], np.int64)
    caps = np.array([1, 2], np.int64)
    assert lib.ea_prefix_coverage(prev.ctypes.data, bad_offs.ctypes.data, 2, caps.ctypes.data, 2,
                                  cov.ctypes.data) == -1
    neg = np.array([-1, 2], np.int64)
    offs = np.array([0, 2, 4], np.int64)
    assert lib.ea_prefix_coverage(prev.ctypes.data, offs.ctypes.data, 2, neg.ctypes.data, 2,
                                  cov.ctypes.data) == -1
    assert not cov.any()
    with pytest.raises(EAError):
        api.prefix_coverage(prev, [0, 2, 4], [-3])


@pytest.mark.parametrize("seed", range(4))
def test_simulation_with_declines_matches_oracle(seed):
    r = np.random.default_rng(40 + seed)
    keys, offs = W.chunk_stream(40 + seed, agents=10, turns=6, start_chunks=24, max_chunks=200,
                                growth_chunks=(2, 12), keep=0.98)
    declined = r.random(len(keys)) < [0.0, 0.2, 0.5, 1.0][seed]
    for K in (0, 1, 150, 600, 1100, 5000):
        want = oracle.lru_reference(keys, K, declined)
        assert np.array_equal(api.lru_simulate(keys, K, declined), want), K
        if seed == 0:  # nothing declined: the one-pass distances agree too
            prev, _ = api.reuse_distances(keys)
            assert np.array_equal((prev >= 0) & (prev < K), want.astype(bool))


def test_simulation_edge_cases():
    assert len(api.lru_simulate(np.zeros((0, 32), np.uint8), 3)) == 0
    same = np.full((3, 32), 1, np.uint8)
    assert list(api.lru_simulate(same, 0)) == [0, 0, 0]
    assert list(api.lru_simulate(same, 1)) == [0, 1, 1]
    assert list(api.lru_simulate(same, 5, [1, 0, 0])) == [0, 0, 1]
    with pytest.raises(EAError):
        api.lru_simulate(same, -1)


def test_full_agent_pool_stream_at_the_tier_capacity():
    # 64 agents x 24 turns, 512-4,096 chunks per request (8k-64k tokens in
    # 16-token chunks), 2.7M references; a 64 GiB tier of 1.5 MiB slots
    keys, offs = W.chunk_stream(W.SEED_WORKLOAD, agents=W.POOL_AGENTS, turns=24,
                                start_chunks=512, max_chunks=4096, growth_chunks=(31, 188),
                                keep=W.POOL_KEEP)
    K = (64 << 30) // (1536 << 10)
    prev, nxt = api.reuse_distances(keys)
    want = oracle.lru_reference(keys, K).astype(bool)
    assert np.array_equal((prev >= 0) & (prev < K), want)
    cov = api.prefix_coverage(prev, offs, [K])[:, 0]
    lead = [int(np.argmin(h)) if not h.all() else len(h)
            for h in (want[offs[j]:offs[j + 1]] for j in range(len(offs) - 1))]
    assert np.array_equal(cov, lead)
    # declining every miss of every other agent's requests
    agent = np.repeat(np.arange(len(offs) - 1) % W.POOL_AGENTS, np.diff(offs))
    declined = (agent % 2 == 1).astype(np.uint8)
    assert np.array_equal(api.lru_simulate(keys, K, declined),
                          oracle.lru_reference(keys, K, declined))


@pytest.mark.parametrize("seed", range(4))
def test_tier_order_simulation_matches_oracle(seed):
    keys, offs = W.chunk_stream(60 + seed, agents=10, turns=7, start_chunks=20, max_chunks=160,
                                growth_chunks=(2, 14), keep=0.9)
    r = np.random.default_rng(70 + seed)
    dec = (r.random(len(offs) - 1) < [0.0, 0.3, 0.7, 1.0][seed]).astype(np.uint8)
    for K in (0, 1, 7, 120, 500, 900, 4000):
        want = oracle.lru_prefix_model(keys, offs, K, dec)
        assert np.array_equal(api.lru_simulate_prefix(keys, offs, K, dec), want), K
        assert np.array_equal(api.lru_simulate_prefix(keys, offs, K), oracle.lru_prefix_model(
            keys, offs, K)), K


def test_tier_order_simulation_edge_cases():
    same = np.full((4, 32), 5, np.uint8)
    # a key repeated inside a request is inserted once and hits twice later
    assert list(api.lru_simulate_prefix(same, [0, 2, 2, 4], 2)) == [0, 0, 2]
    assert list(oracle.lru_prefix_model(same, [0, 2, 2, 4], 2)) == [0, 0, 2]
    assert len(api.lru_simulate_prefix(np.zeros((0, 32), np.uint8), [0], 3)) == 0
    with pytest.raises(EAError):
        api.lru_simulate_prefix(same, [1, 3], 2)
    with pytest.raises(EAError):
        api.lru_simulate_prefix(same, [0, 3, 2], 2)
    with pytest.raises(EAError):
        api.lru_simulate_prefix(same, [0, 3], -2)
