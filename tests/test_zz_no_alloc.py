"""The hashing entry point that allocates nothing, for callers that cannot
call hipMalloc: ea_hash_blocks_device_offsets_noalloc keeps its midstates,
offsets and scan state in fixed device memory.  Called through the C ABI,
its keys and key offsets must equal those of ea_hash_blocks_device_offsets
(and the oracle's) byte for byte, on two calls in a row, the second with a
smaller input; sizes beyond its limits are refused before anything runs."""
import ctypes as C

import numpy as np
import pytest

import oracle
from paper_2609_33762_amd import _native as N
from paper_2609_33762_amd import workloads as W

from gpu_common import need_gpu

pytestmark = pytest.mark.gpu

LIMIT = 1 << 20  # keys and sequences the fixed memory holds


def call(name, torch, toks, offs, b, parents, cap):
    d_tok = torch.as_tensor(toks, device="cuda")
    d_offs = torch.as_tensor(offs, device="cuda")
    out = torch.full((cap, 32), 0xEE, dtype=torch.uint8, device="cuda")
    d_koffs = torch.full((len(offs),), -9, dtype=torch.int64, device="cuda")
    d_par = None if parents is None else torch.as_tensor(parents, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    rc = getattr(N.load(), name)(d_tok.data_ptr(), d_tok.numel(), d_offs.data_ptr(),
                                 len(offs) - 1, b,
                                 None if d_par is None else d_par.data_ptr(), out.data_ptr(),
                                 cap, d_koffs.data_ptr(), C.c_void_p(stream))
    assert rc == N.EA_OK, (name, rc)
    torch.cuda.synchronize()
    return out.cpu().numpy(), d_koffs.cpu().numpy()


@pytest.mark.parametrize("form", [None, "fused"])
@pytest.mark.parametrize("b", [16, 1024])
def test_no_alloc_matches_the_allocating_entry_point(b, form, monkeypatch):
    # also with the fused form forced: its key offsets come from its own
    # kernel and the scan state in the fixed memory
    torch = need_gpu()
    if form:
        monkeypatch.setenv("EA_HASH_CHAIN", form)
    r = W.rng(900 + b)
    cases = [list(r.integers(0, 40 * b, size=3000)), list(r.integers(0, 9 * b, size=37))]
    for k, lengths in enumerate(cases):          # the second call is smaller
        toks, offs = W.sequences(901 + k, lengths)
        par = W.host_bytes(902 + k, 32 * len(lengths)).reshape(-1, 32) if k == 0 else None
        okeys, okoffs = oracle.hash_blocks(toks, offs, b, par)
        cap = len(okeys) + 5
        want, want_off = call("ea_hash_blocks_device_offsets", torch, toks, offs, b, par, cap)
        got, got_off = call("ea_hash_blocks_device_offsets_noalloc", torch, toks, offs, b, par,
                            cap)
        assert np.array_equal(got_off, want_off) and np.array_equal(got_off, okoffs), k
        assert np.array_equal(got, want), k
        assert np.array_equal(got[:len(okeys)], okeys) and (got[len(okeys):] == 0xEE).all(), k


def test_no_alloc_device_errors_and_limits():
    torch = need_gpu()
    # malformed device offsets: reported on the device, nothing written
    d_tok = torch.zeros(64, dtype=torch.int32, device="cuda")
    out = torch.full((8, 32), 0xEE, dtype=torch.uint8, device="cuda")
    d_koffs = torch.full((3,), 5, dtype=torch.int64, device="cuda")
    d_offs = torch.tensor([0, 48, 32], dtype=torch.int64, device="cuda")
    lib = N.load()
    rc = lib.ea_hash_blocks_device_offsets_noalloc(
        d_tok.data_ptr(), 64, d_offs.data_ptr(), 2, 16, None, out.data_ptr(), 8,
        d_koffs.data_ptr(), C.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == N.EA_OK
    torch.cuda.synchronize()
    assert d_koffs[0].item() == -1 and (out.cpu().numpy() == 0xEE).all()
    # beyond the fixed memory: refused on the host, nothing launched
    fake = C.c_void_p(0x10000)
    assert lib.ea_hash_blocks_device_offsets_noalloc(
        fake, 16 * (LIMIT + 1), fake, 1, 16, None, fake, LIMIT + 1, fake, None) == N.EA_EINVAL
    assert lib.ea_hash_blocks_device_offsets_noalloc(
        fake, 16, fake, LIMIT + 1, 16, None, fake, 1, fake, None) == N.EA_EINVAL
    # a limit-sized call is accepted and correct
    n = LIMIT // 64
    toks, offs = W.sequences(905, [1024] * n)
    okeys, okoffs = oracle.hash_blocks(toks, offs, 16)
    got, got_off = call("ea_hash_blocks_device_offsets_noalloc", torch, toks, offs, 16, None,
                        LIMIT)
    assert np.array_equal(got_off, okoffs) and np.array_equal(got, okeys)
