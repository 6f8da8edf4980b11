"""Helpers for the GPU parity tests: build a cache/tier pair on cuda:0 from
seeded inputs and mirror it into the oracle's host arrays."""
import numpy as np
import pytest

import oracle
from paper_2609_33762_amd import api
from paper_2609_33762_amd import workloads as W


def need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a GPU")
    return torch


class Pair:
    """A GPU cache + pinned tier and the oracle's view of the same shape."""

    def __init__(self, num_pages, num_layers, page_tokens, heads, head_dim, elem_bytes,
                 slots, scales=False, seed=0, fp8=False, chunk_pages=1):
        torch = need_gpu()
        self.torch = torch
        self.oshape = oracle.make_shape(num_pages, num_layers, page_tokens, heads, head_dim,
                                        elem_bytes, scales, chunk_pages)
        self.sizes = oracle.sizes(self.oshape)
        self.kv = torch.empty(self.sizes["cache"], dtype=torch.uint8, device="cuda")
        if fp8 or elem_bytes == 1:
            W.fill_random_bytes(self.kv, seed)
        else:
            W.fill_bf16_normal(self.kv, seed)
        self.sc = None
        if scales:
            self.sc = torch.empty(self.sizes["scales"], dtype=torch.uint8, device="cuda")
            W.fill_random_bytes(self.sc, seed + 1000)
        self.cache = api.Cache(self.kv, num_pages, num_layers, page_tokens, heads, head_dim,
                               elem_bytes, scales=self.sc)
        self.tier = api.Tier(self.cache, slots * self.sizes["slot"], chunk_pages=chunk_pages)
        assert self.tier.capacity == slots
        assert self.tier.slot_bytes == self.sizes["slot"]
        # poison the host tier so that untouched slots are recognisable
        self.tier.host_view()[:] = W.host_bytes(seed + 2000, slots * self.sizes["slot"]).reshape(
            slots, -1)
        self.snapshot()

    def snapshot(self):
        """Copy the current GPU/tier images into the oracle's arrays."""
        self.torch.cuda.synchronize()
        self.o_cache = self.kv.cpu().numpy().copy()
        self.o_sc = None if self.sc is None else self.sc.cpu().numpy().copy()
        self.o_tier = self.tier.host_view().copy()

    def o_store(self, ids, slots, mask=None):
        oracle.store_blocks(self.oshape, self.o_cache, self.o_sc, self.o_tier, ids, slots, mask)

    def o_load(self, slots, dst):
        oracle.load_blocks(self.oshape, self.o_tier, self.o_cache, self.o_sc, slots, dst)

    def assert_equal(self, what=""):
        self.torch.cuda.synchronize()
        got_tier = self.tier.host_view()
        if not np.array_equal(got_tier, self.o_tier):
            bad = np.nonzero((got_tier != self.o_tier).any(axis=1))[0]
            raise AssertionError(f"{what}: tier slots differ: {bad[:10]} ({len(bad)} slots)")
        got = self.kv.cpu().numpy()
        if not np.array_equal(got, self.o_cache):
            L, P = self.oshape.num_layers, self.oshape.num_pages
            d = (got.reshape(L, P, -1) != self.o_cache.reshape(L, P, -1)).any(axis=2)
            raise AssertionError(f"{what}: cache pieces differ at (layer, page) {np.argwhere(d)[:10]}")
        if self.sc is not None:
            assert np.array_equal(self.sc.cpu().numpy(), self.o_sc), f"{what}: scales differ"

    def close(self):
        self.tier.close()
        self.cache.close()


# ----------------------------------------------- full-size image checks

POISON = 0xC3


def poison_tier(host, value=POISON):
    """Fill every host slot with one byte value (viewed as 64-bit words)."""
    host.reshape(-1).view(np.uint64)[:] = np.uint64(int.from_bytes(bytes([value]) * 8, "little"))


def assert_poisoned_except(host, written, value=POISON, chunk=256):
    """Every slot not listed in `written` still holds the poison bytes."""
    word = np.uint64(int.from_bytes(bytes([value]) * 8, "little"))
    keep = np.setdiff1d(np.arange(host.shape[0]), np.asarray(written))
    for i in range(0, len(keep), chunk):
        idx = keep[i:i + chunk]
        lo, hi = idx[0], idx[-1] + 1
        if hi - lo == len(idx):   # a contiguous run: compare in place
            ok = (host[lo:hi].reshape(-1).view(np.uint64) == word).all()
        else:
            ok = (host[idx].reshape(-1).view(np.uint64) == word).all()
        assert ok, f"an unwritten slot among {idx[:4]}... lost its poison"


def pages_to_host(torch, kv3, pages, chunk=512):
    """[L][n][piece] host copy of the listed pages, in the listed order."""
    L, _, piece = kv3.shape
    pages = np.asarray(pages)
    out = np.empty((L, len(pages), piece), np.uint8)
    for i in range(0, len(pages), chunk):
        idx = torch.as_tensor(pages[i:i + chunk], device=kv3.device, dtype=torch.int64)
        out[:, i:i + len(idx)] = kv3[:, idx].cpu().numpy()
    return out


def oracle_mini_shape(sh, n):
    return oracle.make_shape(n, sh.num_layers, sh.page_tokens, sh.num_kv_heads, sh.head_dim,
                             sh.elem_bytes, sh.has_scales)


def oracle_slots(sh, mini, mini_scales=None):
    """The oracle's store of pages 0..n-1 of a [L][n][piece] host cache (and
    [L][n][8] scales) into slots 0..n-1: [n][slot_bytes]."""
    n = mini.shape[1]
    o = oracle_mini_shape(sh, n)
    want = np.zeros((n, oracle.sizes(o)["slot"]), np.uint8)
    oracle.store_blocks(o, np.ascontiguousarray(mini).reshape(-1),
                        None if mini_scales is None else np.ascontiguousarray(mini_scales).reshape(-1),
                        want, np.arange(n, dtype=np.int32), np.arange(n, dtype=np.int64))
    return want


def oracle_pages(sh, slots_img, with_scales=False):
    """The oracle's load of slots 0..n-1 into pages 0..n-1 of a fresh host
    cache: [L][n][piece] (and [L][n][8] scales)."""
    n = slots_img.shape[0]
    o = oracle_mini_shape(sh, n)
    out = np.zeros((sh.num_layers, n, sh.piece_bytes), np.uint8)
    sc = np.zeros((sh.num_layers, n, 8), np.uint8) if with_scales else None
    oracle.load_blocks(o, np.ascontiguousarray(slots_img), out.reshape(-1),
                       None if sc is None else sc.reshape(-1), np.arange(n, dtype=np.int64),
                       np.arange(n, dtype=np.int32))
    return (out, sc) if with_scales else out


def changed_pages(torch, kv3, before3, chunk=512):
    """Pages (any layer) whose bytes differ between two [L][P][piece] device
    images."""
    P = kv3.shape[1]
    out = []
    for p0 in range(0, P, chunk):
        p1 = min(P, p0 + chunk)
        d = (kv3[:, p0:p1] != before3[:, p0:p1]).any(dim=2).any(dim=0)
        out.append((torch.nonzero(d).flatten() + p0).cpu().numpy())
    return np.concatenate(out)


def assert_rows_equal(got, want, what):
    if not np.array_equal(got, want):
        bad = np.nonzero((got.reshape(len(got), -1) != want.reshape(len(want), -1)).any(axis=1))[0]
        raise AssertionError(f"{what}: {len(bad)} of {len(got)} rows differ, first {bad[:8]}")
