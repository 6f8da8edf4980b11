"""Workload drivers over the C ABI: the agent pool, dense scattered batches
and the layer-pipelined prefix load.  Each driver only issues library calls
(hash, lookup, admission, alloc, store, load, unpin) and records what it did,
so that the tests can replay every call on the oracle and the benchmark can
time them.  Page contents of the agent pool are a counter-based function of
the block's key (`key_pattern`), so any loaded page can be checked against
its key.
"""
import time
from dataclasses import dataclass, field

import numpy as np

from . import api
from . import workloads as W


# ------------------------------------------------------------ key pattern

_M32 = 0xFFFFFFFF


def key_pattern(torch, keys, words, device, chunk_pages=1):
    """int32 [len(keys) * chunk_pages, words] page contents for blocks with
    these keys: word j of page c of a block whose key starts with the
    little-endian uint32 s is fmix32(s + 0x632BE5AB * c + 0x9E3779B1 * j mod
    2^32) (MurmurHash3's finaliser)."""
    s0 = np.ascontiguousarray(keys[:, :4]).view(np.uint32).astype(np.int64).reshape(-1, 1)
    c = np.arange(chunk_pages, dtype=np.int64).reshape(1, -1)
    seeds = torch.as_tensor(((s0 + c * 0x632BE5AB) & _M32).reshape(-1, 1), device=device)
    j = torch.arange(words, dtype=torch.int64, device=device).reshape(1, -1)
    x = (seeds + j * 0x9E3779B1) & _M32
    x = x ^ (x >> 16)
    x = (x * 0x85EBCA6B) & _M32
    x = x ^ (x >> 13)
    x = (x * 0xC2B2AE35) & _M32
    x = x ^ (x >> 16)
    return (x - ((x >> 31) << 32)).to(torch.int32)  # two's complement view


def write_pages(torch, kv3, pages, content):
    """kv3: uint8 view [L, P, piece]; content int32 [n, L*piece/4]."""
    L, _, piece = kv3.shape
    c = content.view(torch.uint8).view(len(pages), L, piece).permute(1, 0, 2)
    kv3[:, torch.as_tensor(pages, device=kv3.device, dtype=torch.int64)] = c


def read_pages(torch, kv3, pages):
    L, _, piece = kv3.shape
    idx = torch.as_tensor(pages, device=kv3.device, dtype=torch.int64)
    return kv3[:, idx].permute(1, 0, 2).reshape(len(pages), L * piece)


# ------------------------------------------------------------ agent pool

@dataclass
class TurnRecord:
    turn: int
    agent: int
    n_tokens: int
    keys: np.ndarray
    hit: int
    hit_slots: np.ndarray
    save: int
    mask: np.ndarray
    alloc_slots: np.ndarray
    stored: int
    loaded_ok: bool
    load_pages: np.ndarray = field(default=None)
    store_pages: np.ndarray = field(default=None)


class AgentPool:
    """Agents served round-robin; each turn is one request of one agent.

    A block is one host slot: C = tier.chunk_pages pages of T tokens (one
    key per b = C * T tokens).
    A prompt keeps the first floor(0.98 * len) tokens of the agent's previous
    prompt, then fresh tokens up to len' = min(len + U[500, 3000], 65536); an
    agent at 65,536 tokens starts a new task at 8,192.  A turn hashes only
    the blocks after the last unchanged full block (from the cached parent
    key), looks up the prompt's keys, loads the hit prefix into free GPU
    pages, writes the remaining blocks' KV (a function of their keys) into
    other free pages, decides admission, allocates slots, stores the admitted
    blocks and releases the pins.  GPU pages are free again after each turn.

    With load_stream and store_stream, loads and stores run on their own
    streams and a turn does not wait for the previous turn's store: the
    host link carries that store and the next turn's load at once.  The
    library orders transfers that touch the same slot.  GPU pages are the
    caller's: a turn draws its pages apart from the pages of every load and
    store that may still run (an event recorded after each tells), and a
    load starts after the fills issued before it."""

    def __init__(self, torch, cache, tier, kv, shape, policy, agents=W.POOL_AGENTS,
                 seed=W.SEED_WORKLOAD, verify=True, stream=None, time_fill=False,
                 load_stream=None, store_stream=None):
        # time_fill: measure the synthetic KV fill (the stand-in for prefill
        # compute) so that a benchmark can leave it out of the path's time
        self.time_fill = time_fill
        self.fill_seconds = 0.0
        self.torch, self.cache, self.tier, self.kv = torch, cache, tier, kv
        self.sh, self.policy, self.verify = shape, policy, verify
        self.kv3 = kv.view(shape.num_layers, shape.num_pages, shape.piece_bytes)
        self.words = shape.num_layers * shape.piece_bytes // 4
        self.C = tier.chunk_pages  # pages per host slot (one key per C pages)
        self.b = shape.page_tokens * self.C
        self.agents = agents
        self.r = W.rng(seed)
        self.tok_rng = [W.rng(seed * 1000 + a) for a in range(agents)]
        self.prompts = [None] * agents
        self.keys = [np.zeros((0, 32), np.uint8)] * agents
        self.turn_no = 0
        self.stream = stream
        self.load_stream = load_stream if load_stream is not None else stream
        self.store_stream = store_stream if store_stream is not None else stream
        self.overlap = load_stream is not None or store_stream is not None
        self.pending = []  # (event, pages) of loads and stores that may still run
        self.bytes_loaded = 0
        self.bytes_stored = 0

    def _note(self, stream, pages):
        if self.overlap:
            ev = self.torch.cuda.Event()
            ev.record(stream)
            self.pending.append((ev, np.asarray(pages, np.int64)))

    def _busy_pages(self):
        """Pages that a load or store issued earlier may still touch; drains
        them first if they would leave fewer than half the pages free."""
        self.pending = [(e, p) for e, p in self.pending if not e.query()]
        if sum(len(p) for _, p in self.pending) > self.sh.num_pages // 2:
            for e, _ in self.pending:
                e.synchronize()
            self.pending = []
        if not self.pending:
            return np.zeros(0, np.int64)
        return np.concatenate([p for _, p in self.pending])

    def _next_prompt(self, a):
        rng = self.tok_rng[a]
        prev = self.prompts[a]
        if prev is None or len(prev) >= W.POOL_MAX_TOKENS:
            n = W.POOL_START_TOKENS
            p = rng.integers(0, W.VOCAB, size=n, dtype=np.int64).astype(np.int32)
            keep = 0
        else:
            n = min(len(prev) + int(rng.integers(W.POOL_GROWTH[0], W.POOL_GROWTH[1] + 1)),
                    W.POOL_MAX_TOKENS)
            keep = int(np.floor(W.POOL_KEEP * len(prev)))
            fresh = rng.integers(0, W.VOCAB, size=n - keep, dtype=np.int64).astype(np.int32)
            p = np.concatenate([prev[:keep], fresh])
        return p, keep

    def turn(self):
        torch, tier, cache, b, C = self.torch, self.tier, self.cache, self.b, self.C
        a = self.turn_no % self.agents
        t = self.turn_no
        prompt, keep = self._next_prompt(a)
        n_full = len(prompt) // b  # full blocks (chunks of C pages)
        # incremental hash: blocks before the first changed token keep their keys
        j0 = min(keep // b, len(self.keys[a]), n_full)
        parent = self.keys[a][j0 - 1].reshape(1, 32) if j0 > 0 else None
        tail = prompt[j0 * b:]
        new_keys, _ = api.hash_blocks(tail, np.array([0, len(tail)]), b, parent)
        keys = np.concatenate([self.keys[a][:j0], new_keys])[:n_full]
        self.prompts[a], self.keys[a] = prompt, keys

        h, hit_slots = tier.lookup(keys)
        if self.overlap:
            pages = W.distinct(self.r, self.sh.num_pages, n_full * C, exclude=self._busy_pages())
        else:
            pages = W.distinct(self.r, self.sh.num_pages, n_full * C)
        load_pages = pages[:h * C]
        if h:
            if self.overlap and self.load_stream is not None:
                self.load_stream.wait_stream(torch.cuda.current_stream())
            tier.load(cache, hit_slots, load_pages, stream=self.load_stream)
            self.bytes_loaded += h * tier.slot_bytes
            self._note(self.load_stream, load_pages)
        if n_full > h:  # compute (here: synthesise) the KV the tier did not have
            if self.time_fill:
                # nothing of the path runs while the excluded fill is timed
                torch.cuda.synchronize()
                t0 = time.perf_counter()
            step = max(1, 512 // C)
            for c0 in range(h, n_full, step):
                c1 = min(n_full, c0 + step)
                write_pages(torch, self.kv3, pages[c0 * C:c1 * C],
                            key_pattern(torch, keys[c0:c1], self.words, self.kv.device, C))
            if self.time_fill:
                torch.cuda.synchronize()
                self.fill_seconds += time.perf_counter() - t0
        save, mask = tier.admission(self.policy, len(prompt), h * b, a, t, keys)
        _, slots = tier.alloc(keys, mask)
        ok = slots >= 0
        store_pages = pages.reshape(n_full, C)[ok].reshape(-1)
        if ok.any():
            if self.overlap and self.store_stream is not None:
                # the store reads the pages the fill just wrote
                self.store_stream.wait_stream(torch.cuda.current_stream())
            tier.store(cache, store_pages, slots[ok], stream=self.store_stream)
            self.bytes_stored += int(ok.sum()) * tier.slot_bytes
            self._note(self.store_stream, store_pages)
        loaded_ok = True
        if self.verify and h:
            torch.cuda.synchronize()
            step = max(1, 512 // C)
            for c0 in range(0, h, step):
                c1 = min(h, c0 + step)
                want = key_pattern(torch, keys[c0:c1], self.words, self.kv.device, C)
                got = read_pages(torch, self.kv3, load_pages[c0 * C:c1 * C]).view(torch.int32)
                loaded_ok &= bool(torch.equal(got, want))
        if ok.any():
            tier.unpin(slots[ok])
        if h:
            tier.unpin(hit_slots)
        self.turn_no += 1
        return TurnRecord(t, a, len(prompt), keys, h, hit_slots, save, mask, slots,
                          int(ok.sum()), loaded_ok, load_pages, store_pages)


# ------------------------------------------------- dense scattered batches

def non_adjacent_pages(r, num_pages, k):
    """k distinct page ids, no two adjacent."""
    while True:
        p = np.sort(r.choice(num_pages, size=k, replace=False))
        if k < 2 or np.all(np.diff(p) > 1):
            return r.permutation(p)


class DenseScattered:
    """Alternating store and load calls of 1-8 random non-adjacent pages; a
    load reads slots that an earlier store wrote.  Stores allocate slots
    through the tier under fresh random keys (the tier evicts by LRU once
    full); loads pick random resident slots."""

    def __init__(self, cache, tier, shape, seed=W.SEED_WORKLOAD, stream=None):
        self.cache, self.tier, self.sh = cache, tier, shape
        self.r = W.rng(seed)
        self.stream = stream
        self.calls = []

    def call(self, i):
        r, sh = self.r, self.sh
        k = int(r.integers(1, 9))
        if i % 2 == 0:
            pages = non_adjacent_pages(r, sh.num_pages, k)
            keys = r.integers(0, 256, size=(k, 32), dtype=np.uint8)
            _, slots = self.tier.alloc(keys)
            ok = slots >= 0
            self.tier.store(self.cache, pages[ok], slots[ok], stream=self.stream)
            self.tier.unpin(slots[ok])
            rec = ("store", pages[ok], slots[ok])
        else:
            state = self.tier.export()["state"]
            resident = np.nonzero(state == 2)[0]
            k = min(k, len(resident))
            slots = r.choice(resident, size=k, replace=False)
            pages = non_adjacent_pages(r, sh.num_pages, k)
            self.tier.load(self.cache, slots, pages, stream=self.stream)
            rec = ("load", pages, slots)
        self.calls.append(rec)
        return rec


# --------------------------------------------- reference-model capacity report

def stack_report(records, capacity_slots, slot_bytes, curve_bytes=()):
    """Predict the agent pool's host hits with the reuse-distance tool and
    compare them with what the tier measured.

    The reference stream lists, request by request, every full block of the
    prompt in order (the paper's reference model).  Reported, in blocks:
      hits_measured           leading hits the tier returned (sum of h)
      hits_model_full         leading hits of an LRU tier of K_H slots that
                              admits every miss (one-pass reuse distances)
      hits_model_run_declines the same tier with the misses of the requests
                              the run declined left out (Proposition 1's
                              setting)
      hits_model_tier_order   the tier's own order (a lookup promotes only
                              the matched prefix) with the run's declines:
                              this reproduces hits_measured
      declined_new_blocks     new blocks (after the measured hit prefix) of
                              declined requests, and the share of them whose
                              next reuse distance is >= K_H or that are
                              never referenced again (the proposition's
                              condition), the share never referenced again,
                              and the median next reuse distance over K_H of
                              those that are
    and, for each tier size in curve_bytes, the coverage of an LRU tier that
    admits every miss in both orders."""
    lens = np.array([len(r.keys) for r in records], np.int64)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    refs = np.concatenate([r.keys for r in records]) if len(records) else np.zeros((0, 32), np.uint8)
    req_declined = np.array([not r.save for r in records], bool)
    declined = np.repeat(req_declined, lens).astype(np.uint8)
    t0 = time.perf_counter()
    prev, nxt = api.reuse_distances(refs)
    caps = [capacity_slots] + [int(c // slot_bytes) for c in curve_bytes]
    cov = api.prefix_coverage(prev, offs, caps)
    tool_s = time.perf_counter() - t0
    sim = api.lru_simulate(refs, capacity_slots, declined).astype(bool)
    lead = 0
    for j in range(len(records)):
        h = sim[offs[j]:offs[j + 1]]
        lead += int(np.argmin(h)) if not h.all() else len(h)
    tier_order = api.lru_simulate_prefix(refs, offs, capacity_slots, req_declined)
    curve_tier = [api.lru_simulate_prefix(refs, offs, int(c // slot_bytes)).sum()
                  for c in curve_bytes]
    new_mask = np.zeros(len(refs), bool)
    for j, r in enumerate(records):
        if not r.save:
            new_mask[offs[j] + r.hit:offs[j + 1]] = True
    nd = nxt[new_mask]
    far = int(np.sum((nd < 0) | (nd >= capacity_slots)))
    again = nd[nd >= 0]
    return {
        "references": int(len(refs)), "capacity_slots": int(capacity_slots),
        "hits_measured": int(sum(r.hit for r in records)),
        "hits_model_full": int(cov[:, 0].sum()),
        "hits_model_run_declines": lead,
        "hits_model_tier_order": int(tier_order.sum()),
        "hits_tier_order_per_request": tier_order,
        "declined_new_blocks": int(new_mask.sum()),
        "declined_meeting_condition": round(far / max(1, int(new_mask.sum())), 4),
        "declined_never_again": round(int(np.sum(nd < 0)) / max(1, len(nd)), 4),
        "declined_median_next_distance_over_KH":
            round(float(np.median(again)) / capacity_slots, 3) if len(again) else None,
        "coverage_curve_full_admission": {
            str(int(b) >> 30) + "GiB": round(float(cov[:, 1 + i].sum()) / max(1, int(lens.sum())), 4)
            for i, b in enumerate(curve_bytes)},
        "coverage_curve_tier_order": {
            str(int(b) >> 30) + "GiB": round(float(curve_tier[i]) / max(1, int(lens.sum())), 4)
            for i, b in enumerate(curve_bytes)},
        "tool_seconds": round(tool_s, 3),
    }


# ------------------------------------------------------ restore cost (Eq. 2)

def fit_load_cost(nbytes, seconds):
    """Least-squares fit of T_load = bytes / B_eff + tau_load (Eq. 2 with
    n * beta_rank bytes).  Returns (B_eff in bytes/s, tau_load in s, largest
    relative residual)."""
    x = np.asarray(nbytes, np.float64)
    y = np.asarray(seconds, np.float64)
    a, tau = np.polyfit(x, y, 1)
    resid = np.abs(a * x + tau - y) / y
    return 1.0 / a, tau, float(resid.max())


def load_cost_sweep(torch, cache, tier, sh, sizes, stream, rng, reps=None):
    """Loads of n random resident slots into random free pages for each n in
    `sizes` (slots 0..max(sizes)-1 of `tier` must hold stored chunks).
    Returns rows [tokens, bytes, device ms, end-to-end ms], each the median
    over its repetitions: device time between HIP events on the load's
    stream, end to end from the call to completion on the host clock."""
    C = tier.chunk_pages
    top = max(sizes)
    rows = []
    for n in sizes:
        k = reps or (40 if n * C <= 64 else (10 if n * C <= 512 else 5))
        dev_ms, wall_ms = [], []
        for _ in range(k):
            slots = W.distinct(rng, top, n)
            dst = W.distinct(rng, sh.num_pages, n * C)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            e0.record(stream)
            tier.load(cache, slots, dst, stream=stream)
            e1.record(stream)
            e1.synchronize()
            wall_ms.append((time.perf_counter() - t0) * 1e3)
            dev_ms.append(e0.elapsed_time(e1))
        rows.append([n * C * sh.page_tokens, n * tier.slot_bytes, float(np.median(dev_ms)),
                     float(np.median(wall_ms))])
    return rows
