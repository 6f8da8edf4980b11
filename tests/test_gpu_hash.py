"""GPU parity of the chained prefix-block keys against the oracle: ragged
sequences, several block sizes, parents, many chains at once, the workload
sizes (tiny, one Qwen3 agent turn, the 64k-token layered prefix) and the
device-pointer variant."""
import numpy as np
import pytest

import oracle
from paper_2609_33762_amd import api
from paper_2609_33762_amd import workloads as W

from gpu_common import need_gpu

pytestmark = pytest.mark.gpu


def check(lengths, b, parents=False, seed=0):
    need_gpu()
    toks, offs = W.sequences(seed, lengths)
    par = W.host_bytes(seed + 1, 32 * len(lengths)).reshape(-1, 32) if parents else None
    keys, koffs = api.hash_blocks(toks, offs, b, par)
    okeys, okoffs = oracle.hash_blocks(toks, offs, b, par)
    assert np.array_equal(koffs, okoffs)
    if not np.array_equal(keys, okeys):
        bad = np.nonzero((keys != okeys).any(axis=1))[0]
        raise AssertionError(f"{len(bad)} keys differ, first {bad[:8]}")
    return keys, koffs


def test_tiny_workload():
    check([512] * 4, 16, seed=W.SEED_TOKENS)


@pytest.mark.parametrize("b", [16, 32, 1024])
def test_ragged_lengths_and_parents(b):
    lengths = [0, b - 1, b, b + 1, 7 * b + 3, 1, 3 * b]
    check(lengths, b, seed=b)
    check(lengths, b, parents=True, seed=b + 1)


def test_many_chains_span_several_waves():
    r = W.rng(5)
    check(list(r.integers(0, 900, size=300)), 16, parents=True, seed=5)


def test_one_qwen3_turn():
    # the store refill (32k tokens) and the cached prefix (24k) of one turn
    check([32000, 24000], 16, seed=W.SEED_TOKENS)


def test_64k_prefix_chain():
    keys, _ = check([65536], 16, seed=9)
    assert keys.shape == (4096, 32)


def test_device_variant():
    torch = need_gpu()
    toks, offs = W.sequences(3, [100, 0, 513, 1024])
    d_tok = torch.as_tensor(toks, device="cuda")
    okeys, okoffs = oracle.hash_blocks(toks, offs, 16)
    out = torch.zeros((len(okeys), 32), dtype=torch.uint8, device="cuda")
    koffs = api.hash_blocks_device(d_tok, offs, 16, out)
    torch.cuda.synchronize()
    assert np.array_equal(koffs, okoffs)
    assert np.array_equal(out.cpu().numpy(), okeys)


def test_incremental_hash_from_cached_parent():
    # a prompt that repeats an earlier one hashes only its new blocks
    toks, offs = W.sequences(4, [4096])
    full, _ = oracle.hash_blocks(toks, offs, 16)
    k = 200
    tail, _ = api.hash_blocks(toks[16 * k:], np.array([0, 4096 - 16 * k]), 16,
                              parents=full[k - 1].reshape(1, 32))
    assert np.array_equal(tail, full[k:])


@pytest.mark.parametrize("b", [16, 48])
def test_full_int32_range_tokens(b):
    # token values are hashed as the bytes of their two's-complement value:
    # negative ids and both extremes included
    need_gpu()
    r = W.rng(77 + b)
    lengths = [5 * b + 7, 0, 3 * b, 11 * b + 1]
    toks = r.integers(-2**31, 2**31, size=sum(lengths), dtype=np.int64).astype(np.int32)
    toks[:4] = [-2**31, 2**31 - 1, -1, 0]
    offs = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    keys, koffs = api.hash_blocks(toks, offs, b)
    okeys, okoffs = oracle.hash_blocks(toks, offs, b)
    assert np.array_equal(koffs, okoffs) and np.array_equal(keys, okeys)


def test_device_calls_back_to_back():
    # asynchronous calls reuse their offset and midstate buffers in turn:
    # four calls in flight on one stream, different inputs, all correct
    torch = need_gpu()
    cases = [[100, 0, 513, 1024], [4096], [16] * 300, [2000, 31, 777]]
    outs, want = [], []
    for c, lengths in enumerate(cases):
        toks, offs = W.sequences(40 + c, lengths)
        okeys, _ = oracle.hash_blocks(toks, offs, 16)
        d_tok = torch.as_tensor(toks, device="cuda")
        out = torch.zeros((len(okeys), 32), dtype=torch.uint8, device="cuda")
        api.hash_blocks_device(d_tok, offs, 16, out)
        outs.append((d_tok, out))
        want.append(okeys)
    torch.cuda.synchronize()
    for (_, out), okeys in zip(outs, want):
        assert np.array_equal(out.cpu().numpy(), okeys)


@pytest.mark.parametrize("form", ["pair", "lane", "split", "fused"])
def test_every_chain_form(form, monkeypatch):
    # the chained compression runs two lanes per sequence, one lane per
    # sequence (large batches), a workgroup of two waves per four sequences
    # (up to eight sequences per compute unit), or, for the largest batches, one lane
    # per sequence for token blocks and chain alike (fused); each form forced
    # on ragged chains, parents, chunk-sized blocks, a long chain and the
    # extreme token values
    monkeypatch.setenv("EA_HASH_CHAIN", form)
    r = W.rng(90 + len(form))
    check(list(r.integers(0, 900, size=300)), 16, parents=True, seed=91)
    check([0, 15, 16, 17, 1024 * 3 + 5, 2048], 1024, parents=True, seed=92)
    check([65536], 16, seed=93)
    lengths = [5 * 16 + 7, 0, 48, 11 * 16 + 1]
    toks = r.integers(-2**31, 2**31, size=sum(lengths), dtype=np.int64).astype(np.int32)
    toks[:4] = [-2**31, 2**31 - 1, -1, 0]
    offs = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    keys, koffs = api.hash_blocks(toks, offs, 16)
    okeys, okoffs = oracle.hash_blocks(toks, offs, 16)
    assert np.array_equal(koffs, okoffs) and np.array_equal(keys, okeys)


def test_batch_past_the_one_lane_threshold():
    # more sequences than two-lane waves fit one per SIMD (32 per SIMD):
    # the library picks the one-lane chain by itself; ragged lengths, parents;
    # past 256 sequences per compute unit it picks the fused form
    r = W.rng(95)
    check(list(r.integers(0, 160, size=40000)), 16, parents=True, seed=95)
    check([64] * 40000, 16, seed=96)
    check(list(r.integers(0, 400, size=70000)), 16, parents=True, seed=97)


@pytest.mark.parametrize("form", ["pair", "lane", "split"])
def test_64_bit_offsets(form, monkeypatch):
    # offsets travel as 32-bit values when they fit; the 64-bit form (used
    # past 2^31 tokens or keys) forced on ragged sequences, both entry points
    torch = need_gpu()
    monkeypatch.setenv("EA_HASH_OFFSETS", "64")
    monkeypatch.setenv("EA_HASH_CHAIN", form)
    r = W.rng(97)
    check(list(r.integers(0, 700, size=200)), 16, parents=True, seed=97)
    check([0, 1023, 1024, 5000], 1024, seed=98)
    toks, offs = W.sequences(99, [100, 0, 513, 1024, 16])
    d_tok = torch.as_tensor(toks, device="cuda")
    okeys, okoffs = oracle.hash_blocks(toks, offs, 16)
    out = torch.zeros((len(okeys), 32), dtype=torch.uint8, device="cuda")
    koffs = api.hash_blocks_device(d_tok, offs, 16, out)
    torch.cuda.synchronize()
    assert np.array_equal(koffs, okoffs)
    assert np.array_equal(out.cpu().numpy(), okeys)


def test_few_long_chains_take_the_split_form():
    # up to eight sequences per compute unit the library picks the two-wave
    # form by itself: ragged long chains with parents, a chain of one key,
    # empty sequences
    r = W.rng(101)
    lengths = [int(x) for x in r.integers(0, 20000, size=40)] + [16, 0, 15]
    check(lengths, 16, parents=True, seed=101)


@pytest.mark.parametrize("lengths", [
    [16 * 40, 0, 16 * 3, 16 * 7 + 5],         # the longest chain in row 0, an empty row
    [16, 16 * 2, 0, 16 * 50 + 3],             # the longest in row 3
    [16 * 9, 16 * 9, 16 * 9, 16 * 9, 16 * 2],  # a second workgroup with one row
    [0, 0, 0, 15, 16 * 12, 0, 16],            # rows without a key, two workgroups
])
def test_split_rows_of_unequal_length(lengths, monkeypatch):
    # the two-wave form carries four sequences per workgroup, one per row of
    # 16 lanes, each row running as many keys as the longest: every key of
    # every row, with parents, equals the oracle's
    monkeypatch.setenv("EA_HASH_CHAIN", "split")
    check(lengths, 16, parents=True, seed=120 + len(lengths))
    check(lengths, 16, seed=130 + len(lengths))


@pytest.mark.parametrize("extra", [0, 1])
def test_split_form_threshold(extra):
    # eight sequences per compute unit (the last batch of the two-wave form)
    # and one more (the first of the two-lane form), ragged chains of up to
    # 40 keys with parents
    torch = need_gpu()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    r = W.rng(102 + extra)
    lengths = [int(x) for x in r.integers(0, 640, size=8 * cus + extra)]
    check(lengths, 16, parents=True, seed=102 + extra)


@pytest.mark.parametrize("form", ["lane", "split"])
@pytest.mark.parametrize("b", [32, 1024])
def test_midstate_forms(form, b, monkeypatch):
    # the token blocks of a key are compressed by one lane, or for few keys
    # of several blocks by a workgroup of two waves per four keys; each form
    # forced on ragged sequences with parents, a single key (three rows of
    # its workgroup past the last key), and many keys
    monkeypatch.setenv("EA_HASH_MID", form)
    r = W.rng(110 + b)
    check([0, b - 1, b, b + 1, 7 * b + 3, 3 * b], b, parents=True, seed=111)
    check([b], b, seed=112)
    check(list(r.integers(0, 20 * b, size=30)), b, parents=True, seed=113)


@pytest.mark.parametrize("b,per_cu", [(32, 8), (64, 16), (1024, 16)])
@pytest.mark.parametrize("extra", [0, 1])
def test_midstate_split_threshold(b, per_cu, extra):
    # the last batch of keys the library gives the two-wave midstate form
    # (8 keys per compute unit for two-block keys, 16 from four blocks) and
    # one key more (the first of the one-lane form): ragged sequences with
    # parents, so that the four rows of a workgroup span several sequences
    torch = need_gpu()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    r = W.rng(140 + b + extra)
    n_keys = per_cu * cus + extra
    lengths, total = [], 0
    while total < n_keys:  # 0..6 keys and a ragged tail per sequence
        k = min(int(r.integers(0, 7)), n_keys - total)
        lengths.append(k * b + int(r.integers(0, b)))
        total += k
    check(lengths, b, parents=True, seed=141 + extra)


def test_longest_contexts():
    # the paper's longest contexts: the 262,144-token maximum of the serving
    # configuration and the 238,105-token prompt it reports, in 16-token
    # blocks and in 1,024-token chunks (ragged tails)
    check([262144], 16, seed=121)
    check([238105], 16, seed=122)
    check([238105, 262144], 1024, parents=True, seed=123)


def device_offsets_case(torch, lengths, b, seed, parents=False, keys_capacity=None,
                        tokens_pad=0):
    toks, offs = W.sequences(seed, lengths)
    par = W.host_bytes(seed + 1, 32 * len(lengths)).reshape(-1, 32) if parents else None
    okeys, okoffs = oracle.hash_blocks(toks, offs, b, par)
    d_tok = torch.as_tensor(np.concatenate([toks, np.zeros(tokens_pad, np.int32)]),
                            device="cuda")
    d_offs = torch.as_tensor(offs, device="cuda")
    cap = len(okeys) if keys_capacity is None else keys_capacity
    out = torch.full((max(cap, 1), 32), 0xEE, dtype=torch.uint8, device="cuda")
    d_koffs = torch.full((len(offs),), -7, dtype=torch.int64, device="cuda")
    d_par = None if par is None else torch.as_tensor(par, device="cuda")
    api.hash_blocks_device_offsets(d_tok, d_offs, b, out[:cap] if cap else out[:0], d_koffs,
                                   d_parents=d_par)
    return okeys, okoffs, out, d_koffs


@pytest.mark.parametrize("b", [16, 32, 1024])
def test_device_offsets_variant(b):
    # sequence offsets on the device too: the key offsets come from a scan
    # kernel; ragged sequences, empty ones, parents, tokens past the last
    # sequence (ignored)
    torch = need_gpu()
    lengths = [0, b - 1, b, b + 1, 7 * b + 3, 1, 3 * b, 0]
    for parents in (False, True):
        okeys, okoffs, out, d_koffs = device_offsets_case(torch, lengths, b, 60 + b, parents,
                                                          tokens_pad=5 * b)
        torch.cuda.synchronize()
        assert np.array_equal(d_koffs.cpu().numpy(), okoffs)
        assert np.array_equal(out[:len(okeys)].cpu().numpy(), okeys)
        assert (out[len(okeys):].cpu().numpy() == 0xEE).all()


def test_device_offsets_many_sequences_and_forms(monkeypatch):
    # more sequences than the scan's 1,024 threads (several runs each), and
    # every chain form
    torch = need_gpu()
    r = W.rng(71)
    lengths = list(r.integers(0, 300, size=5000))
    for form in ["pair", "lane", "split", "fused", None]:
        if form:
            monkeypatch.setenv("EA_HASH_CHAIN", form)
        else:
            monkeypatch.delenv("EA_HASH_CHAIN", raising=False)
        okeys, okoffs, out, d_koffs = device_offsets_case(torch, lengths, 16, 72, True)
        torch.cuda.synchronize()
        assert np.array_equal(d_koffs.cpu().numpy(), okoffs), form
        assert np.array_equal(out.cpu().numpy()[:len(okeys)], okeys), form


def test_device_offsets_batch_workload_size():
    # the batch of the hash benchmark: 65,536 sequences of 256 tokens
    torch = need_gpu()
    n, L = 65536, 256
    r = W.rng(73)
    toks = r.integers(0, W.VOCAB, size=n * L, dtype=np.int64).astype(np.int32)
    offs = np.arange(0, n * L + 1, L, dtype=np.int64)
    okeys, okoffs = oracle.hash_blocks(toks, offs, 16)
    d_tok = torch.as_tensor(toks, device="cuda")
    out = torch.zeros((len(okeys), 32), dtype=torch.uint8, device="cuda")
    d_koffs = torch.zeros(n + 1, dtype=torch.int64, device="cuda")
    api.hash_blocks_device_offsets(d_tok, torch.as_tensor(offs, device="cuda"), 16, out, d_koffs)
    torch.cuda.synchronize()
    assert np.array_equal(d_koffs.cpu().numpy(), okoffs)
    assert np.array_equal(out.cpu().numpy(), okeys)


@pytest.mark.parametrize("b", [16, 64])
@pytest.mark.parametrize("form", [None, "fused"])
def test_device_offsets_errors_are_reported_on_the_device(form, b, monkeypatch):
    # malformed device offsets or too small an output: key_offsets[0] = -1
    # and no key is written; a later good call on the same stream works;
    # also with the fused form, which derives the offsets in its own kernel,
    # and with keys of four blocks (the two-wave midstate form)
    torch = need_gpu()
    if form:
        monkeypatch.setenv("EA_HASH_CHAIN", form)
    m = b // 16
    cases = [
        ([0, 32, 16, 48], 64, None),     # a decrease
        ([-16, 0, 32], 64, None),        # a negative start
        ([0, 32, 80], 64, None),         # past the 64 tokens given
        ([0, 32, 64], 64, 3),            # 4 keys, room for 3
    ]
    for offs, n_tok, cap in cases:
        offs = [m * o for o in offs]
        d_tok = torch.zeros(m * n_tok, dtype=torch.int32, device="cuda")
        out = torch.full((cap or 8, 32), 0xEE, dtype=torch.uint8, device="cuda")
        d_koffs = torch.full((len(offs),), 5, dtype=torch.int64, device="cuda")
        api.hash_blocks_device_offsets(d_tok, torch.tensor(offs, dtype=torch.int64,
                                                           device="cuda"), b, out, d_koffs)
        torch.cuda.synchronize()
        assert d_koffs[0].item() == -1, offs
        assert (out.cpu().numpy() == 0xEE).all(), offs
    okeys, okoffs, out, d_koffs = device_offsets_case(torch, [64, 48], 16, 74)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy(), okeys)


@pytest.mark.parametrize("b", [64, 1024])
def test_device_offsets_room_for_more_keys(b):
    # device offsets with room for 37 keys more than the sequences hold: the
    # kernels are sized for the room, and every key slot past the last key
    # stays untouched
    torch = need_gpu()
    lengths = [3 * b + 5, 0, b, 7 * b - 1, 2 * b]
    n = sum(x // b for x in lengths)
    okeys, okoffs, out, d_koffs = device_offsets_case(torch, lengths, b, 80 + b, parents=True,
                                                      keys_capacity=n + 37)
    torch.cuda.synchronize()
    assert np.array_equal(d_koffs.cpu().numpy(), okoffs)
    got = out.cpu().numpy()
    assert np.array_equal(got[:n], okeys)
    assert (got[n:] == 0xEE).all()


def test_device_offsets_no_sequences():
    torch = need_gpu()
    d_koffs = torch.full((1,), 9, dtype=torch.int64, device="cuda")
    out = torch.zeros((1, 32), dtype=torch.uint8, device="cuda")
    api.hash_blocks_device_offsets(torch.zeros(16, dtype=torch.int32, device="cuda"),
                                   torch.zeros(1, dtype=torch.int64, device="cuda"), 16, out,
                                   d_koffs)
    torch.cuda.synchronize()
    assert d_koffs.item() == 0 and not out.any()


def test_device_variant_size_checks():
    # the sizes of device buffers cross the boundary: too few tokens or too
    # small an output is refused before anything runs
    torch = need_gpu()
    from paper_2609_33762_amd import _native as N
    import ctypes as C
    d_tok = torch.zeros(40, dtype=torch.int32, device="cuda")
    out = torch.full((2, 32), 0xEE, dtype=torch.uint8, device="cuda")
    with pytest.raises(ValueError):
        api.hash_blocks_device(d_tok, np.array([0, 48]), 16, out)     # 48 > 40 tokens
    with pytest.raises(ValueError):
        api.hash_blocks_device(d_tok, np.array([0, 16, 40]), 16, out[:1])  # 2 keys, room 1
    offs = (C.c_int64 * 2)(0, 48)
    koffs = (C.c_int64 * 2)()
    rc = N.load().ea_hash_blocks_device(d_tok.data_ptr(), 40, offs, 1, 16, None,
                                        out.data_ptr(), 2, koffs, None)
    assert rc == N.EA_EINVAL
    torch.cuda.synchronize()
    assert (out.cpu().numpy() == 0xEE).all()
