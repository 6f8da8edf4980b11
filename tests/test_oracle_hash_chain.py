"""Pins of the oracle's chained prefix-block keys.

The paper fixes the properties (section 2 'Exact-prefix reuse', section 3.2
and App. 'Prefix coverage from a reference stream'): a full chunk's key hashes
its entire preceding context, so equal text after a different prefix gets a
different key and an early edit rekeys every later chunk; only full chunks
have keys.  The byte serialisation is this library's reading (tokens as
little-endian int32, then the previous key); hashlib applied to that message
checks the composition independently of the oracle's SHA-256.
"""
import hashlib

import numpy as np
import pytest

import oracle


def _chain_hashlib(tokens, b, parent=b"\0" * 32):
    keys = []
    prev = parent
    for i in range(len(tokens) // b):
        msg = np.asarray(tokens[i * b:(i + 1) * b], dtype="<i4").tobytes() + prev
        prev = hashlib.sha256(msg).digest()
        keys.append(prev)
    return keys


@pytest.mark.parametrize("b", [1, 7, 16, 32, 1024])
def test_composition_matches_hashlib(b):
    rng = np.random.default_rng(b)
    lens = [0, b - 1 if b > 1 else 0, b, 3 * b + (b // 2), 5 * b]
    toks = [rng.integers(-2**31, 2**31, size=n, dtype=np.int64).astype(np.int32) for n in lens]
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    flat = np.concatenate(toks) if sum(lens) else np.zeros(0, np.int32)
    parents = rng.integers(0, 256, size=(len(lens), 32), dtype=np.uint8)
    keys, koffs = oracle.hash_blocks(flat, offs, b, parents)
    assert list(koffs) == list(np.concatenate([[0], np.cumsum([n // b for n in lens])]))
    for s, t in enumerate(toks):
        ref = _chain_hashlib(t, b, parents[s].tobytes())
        got = [keys[k].tobytes() for k in range(koffs[s], koffs[s + 1])]
        assert got == ref


def _keys(tokens, b=16, parent=None):
    offs = np.array([0, len(tokens)], np.int64)
    k, _ = oracle.hash_blocks(np.asarray(tokens, np.int32), offs, b,
                              None if parent is None else parent.reshape(1, 32))
    return k


def test_zero_root_equals_explicit_zero_parent():
    rng = np.random.default_rng(3)
    t = rng.integers(0, 32000, 160).astype(np.int32)
    assert np.array_equal(_keys(t), _keys(t, parent=np.zeros(32, np.uint8)))


def test_equal_prefixes_give_equal_chains():
    rng = np.random.default_rng(4)
    a = rng.integers(0, 32000, 512).astype(np.int32)
    b = a.copy()
    b[300:] = rng.integers(0, 32000, 212)
    ka, kb = _keys(a), _keys(b)
    # blocks 0..17 are identical token-for-token
    assert np.array_equal(ka[:300 // 16], kb[:300 // 16])


@pytest.mark.parametrize("j", [0, 15, 16, 200, 511])
def test_changing_one_token_rekeys_exactly_the_later_blocks(j):
    rng = np.random.default_rng(5)
    a = rng.integers(0, 32000, 512).astype(np.int32)
    b = a.copy()
    b[j] = (b[j] + 1) % 32000
    ka, kb = _keys(a), _keys(b)
    for i in range(512 // 16):
        same = np.array_equal(ka[i], kb[i])
        assert same == (i < j // 16), i


def test_same_block_after_different_prefix_gets_different_key():
    rng = np.random.default_rng(6)
    block = rng.integers(0, 32000, 16).astype(np.int32)
    p1 = rng.integers(0, 32000, 32).astype(np.int32)
    p2 = p1.copy()
    p2[0] += 1
    k1 = _keys(np.concatenate([p1, block]))
    k2 = _keys(np.concatenate([p2, block]))
    assert not np.array_equal(k1[2], k2[2])


def test_partial_tail_changes_nothing_and_gets_no_key():
    rng = np.random.default_rng(7)
    a = rng.integers(0, 32000, 16 * 9 + 5).astype(np.int32)
    b = a.copy()
    b[-5:] = 0
    ka, kb = _keys(a), _keys(b)
    assert ka.shape == (9, 32)
    assert np.array_equal(ka, kb)


def test_continuation_from_parent_equals_tail_of_full_chain():
    rng = np.random.default_rng(8)
    a = rng.integers(0, 32000, 16 * 40).astype(np.int32)
    full = _keys(a)
    for k in [1, 7, 39]:
        tail = _keys(a[16 * k:], parent=full[k - 1])
        assert np.array_equal(tail, full[k:])


def test_empty_inputs():
    keys, offs = oracle.hash_blocks(np.zeros(0, np.int32), np.array([0], np.int64), 16)
    assert keys.shape == (0, 32) and list(offs) == [0]
    keys, offs = oracle.hash_blocks(np.zeros(0, np.int32), np.array([0, 0, 0], np.int64), 16)
    assert keys.shape == (0, 32) and list(offs) == [0, 0, 0]


def test_invalid_arguments_rejected():
    with pytest.raises(oracle.OracleError):
        oracle.hash_blocks(np.zeros(4, np.int32), np.array([0, 4], np.int64), 0)
    with pytest.raises(oracle.OracleError):
        oracle.hash_blocks(np.zeros(4, np.int32), np.array([3, 1], np.int64), 1)
