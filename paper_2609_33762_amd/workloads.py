"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke
check.  This module holds shapes and random-number recipes only; none of the
offload path's arithmetic lives here.

The five workloads follow the shapes of the paper's serving setups
(Qwen3-Coder-30B-A3B: 48 layers, 4 KV heads, head_dim 128, bf16; the dense
Qwen2.5-Coder-32B family: 8 KV heads) with 16-token pages.  The paper's own
traffic (SWE-bench Verified agent trajectories) is not available; the agent
pool generator stands in for it with the paper's reported shape: prompts that
repeat about 98% of the agent's previous prompt and grow turn by turn.
"""
from dataclasses import dataclass

import numpy as np

VOCAB = 32000
# seeds per role, fixed for every workload
SEED_DATA, SEED_TOKENS, SEED_IDS, SEED_WORKLOAD = 0, 1, 2, 3


@dataclass(frozen=True)
class Shape:
    name: str
    num_layers: int
    num_kv_heads: int
    head_dim: int
    elem_bytes: int
    page_tokens: int
    num_pages: int
    has_scales: bool = False
    dtype: str = "bf16"

    @property
    def piece_bytes(self):  # bytes of one (layer, page): K and V
        return 2 * self.page_tokens * self.num_kv_heads * self.head_dim * self.elem_bytes

    @property
    def cache_bytes(self):
        return self.num_layers * self.num_pages * self.piece_bytes


# Tiny: 256 pages, 2 layers, 2 KV heads, head_dim 64, bf16; 32 pages stored
# then loaded into 32 other free pages; 4 sequences of 512 tokens hashed.
TINY = Shape("tiny", 2, 2, 64, 2, 16, 256)
TINY_TIER_SLOTS = 64
# Qwen3-30B-A3B-shaped KV, one agent turn: 20,000-page cache, 16 GiB tier,
# store a 32k-token refill (2,000 pages), load a 24k-token prefix (1,500).
QWEN3 = Shape("qwen3_30b_a3b_turn", 48, 4, 128, 2, 16, 20000)
QWEN3_TIER_BYTES = 16 << 30
QWEN3_STORE_PAGES = 2000
QWEN3_LOAD_PAGES = 1500
# The same model's KV on one rank of TP8 (1 KV head: 24 KiB per token) with
# the paper's host chunk of 1,024 tokens = 64 pages (24 MiB per slot).
QWEN3_TP8 = Shape("qwen3_30b_a3b_tp8_shard", 48, 1, 128, 2, 16, 20000)
CHUNK_PAGES = 64
# Agent pool: same KV shape, 64 agents, 64 GiB tier.
POOL_TIER_BYTES = 64 << 30
POOL_AGENTS = 64
POOL_START_TOKENS = 8192
POOL_MAX_TOKENS = 65536
POOL_GROWTH = (500, 3000)
POOL_KEEP = 0.98
# Dense KV, small scattered batches: 32 layers, 8 KV heads, head_dim 128.
DENSE = Shape("dense_scattered", 32, 8, 128, 2, 16, 4096)
DENSE_TIER_SLOTS = 4096
DENSE_CALLS = 10000
# Layer-pipelined fp8 prefix load: 64k tokens = 4,096 pages, per-page scales.
LAYERED = Shape("layered_fp8", 48, 4, 128, 1, 16, 8192, has_scales=True, dtype="fp8_e4m3")
LAYERED_PREFIX_PAGES = 4096
# The same prefix on one rank of TP8: 1 KV head, 4 KiB pieces.
LAYERED_TP8 = Shape("layered_fp8_tp8_shard", 48, 1, 128, 1, 16, 8192, has_scales=True,
                    dtype="fp8_e4m3")


def rng(seed):
    return np.random.default_rng(seed)


def tokens(seed, n):
    """Token ids uniform in [0, 32000)."""
    return rng(seed).integers(0, VOCAB, size=n, dtype=np.int64).astype(np.int32)


def sequences(seed, lengths):
    """Concatenated token sequences and their int64 offsets."""
    lengths = list(lengths)
    flat = tokens(seed, int(sum(lengths)))
    offs = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    return flat, offs


def distinct(r, high, k, exclude=None):
    """k distinct integers in [0, high) avoiding `exclude`."""
    if exclude is None or len(exclude) == 0:
        return r.choice(high, size=k, replace=False)
    pool = np.setdiff1d(np.arange(high), np.asarray(exclude))
    return r.choice(pool, size=k, replace=False)


def fill_bf16_normal(t_bytes, seed, chunk_elems=1 << 28):
    """Fill a CUDA uint8 tensor with bf16 N(0,1) values from a seeded
    generator on its device (chunked, so no large temporaries)."""
    import torch
    g = torch.Generator(device=t_bytes.device)
    g.manual_seed(seed)
    view = t_bytes.view(torch.bfloat16)
    n = view.numel()
    for s in range(0, n, chunk_elems):
        e = min(n, s + chunk_elems)
        view[s:e].copy_(torch.randn(e - s, generator=g, device=t_bytes.device,
                                    dtype=torch.float32).to(torch.bfloat16))


def fill_random_bytes(t_bytes, seed, chunk=1 << 30):
    """Fill a CUDA uint8 tensor with uniform random bytes (fp8 payloads and
    scales, NaN encodings included)."""
    import torch
    g = torch.Generator(device=t_bytes.device)
    g.manual_seed(seed)
    n = t_bytes.numel()
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        t_bytes[s:e].copy_(torch.randint(0, 256, (e - s,), generator=g, device=t_bytes.device,
                                         dtype=torch.int32).to(torch.uint8))


def host_bytes(seed, n):
    """Uniform random bytes on the host (small CPU-side cases)."""
    return rng(seed).integers(0, 256, size=n, dtype=np.uint8)


def chunk_stream(seed, agents, turns, start_chunks, max_chunks, growth_chunks, keep):
    """A synthetic chunk reference stream with the agent pool's shape, in
    chunk units and without tokens: agents are served round-robin; a request
    keeps the first floor(keep * len) chunk keys of the agent's previous
    request and continues with fresh random keys up to
    min(len + U[growth_chunks], max_chunks) chunks; an agent at max_chunks
    starts a new task of start_chunks fresh chunks.  Returns (keys uint8
    [n, 32], req_off int64 [agents * turns + 1])."""
    r = rng(seed)
    ctx = [r.integers(0, 256, size=(start_chunks, 32), dtype=np.uint8) for _ in range(agents)]
    first = [True] * agents
    out, offs = [], [0]
    for _ in range(turns):
        for a in range(agents):
            c = ctx[a]
            if first[a]:
                first[a] = False
            elif len(c) >= max_chunks:
                c = r.integers(0, 256, size=(start_chunks, 32), dtype=np.uint8)
            else:
                n = min(len(c) + int(r.integers(growth_chunks[0], growth_chunks[1] + 1)),
                        max_chunks)
                k = int(np.floor(keep * len(c)))
                c = np.concatenate([c[:k], r.integers(0, 256, size=(n - k, 32), dtype=np.uint8)])
            ctx[a] = c
            out.append(c)
            offs.append(offs[-1] + len(c))
    keys = np.concatenate(out) if out else np.zeros((0, 32), np.uint8)
    return keys, np.asarray(offs, np.int64)

