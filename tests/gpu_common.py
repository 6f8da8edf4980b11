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
