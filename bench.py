"""Benchmark: one agent turn of KV offloading on the Qwen3-30B-A3B KV shape.

Workload (48 layers, 4 KV heads, head_dim 128, bf16 = 96 KiB per token,
16-token pages of 1.5 MiB, 20,000-page GPU cache = 29.3 GiB, 16 GiB pinned
host tier = 10,922 slots).  The turn's prompt is a cached 24k-token prefix
followed by a fresh 32k-token refill.  One step is one pass of the whole path
for one turn:
  hash     chained keys of the whole 56k-token prompt (one chain: the
           refill's keys depend on the prefix);
  lookup   consecutive-prefix lookup (1,500 hits, up to the refill);
  load     the 1,500 prefix pages from the host tier into free GPU pages;
  admit    write admission for the request and deduplication of its keys;
  alloc    2,000 host slots (lowest free, LRU eviction once the tier is full);
  store    the 2,000 refill pages from HBM into the host tier;
  unpin    release the lookup and allocation pins.
Store and load run on two streams so the host link carries both directions.
Every step hashes and stores a fresh refill (new tokens), so the tier fills
and starts evicting after five steps, as a serving run would.

Prints one JSON line; details go to stderr and bench_out/bench_detail.json.

Other modes:
  --workload W             the other workloads (agent pool, dense scattered
                           calls, layered fp8 load, tiny, hash, restore-cost
                           fit, TP8 shard, chunked pool, transfer plans)
  --isolated-only          set-up plus the isolated kernel measurements only
  --summarize-profiles D   turn the rocprofv3 CSVs of the default command
                           under D into the summaries in profiles/
  --summarize-plans D      the same for the two transfer plans
  --summarize-hash D       the hash workload's kernel trace under D
"""
import argparse
import csv
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

GB = 1e9
HBM_PEAK_GBS = 8000.0
KERNEL_SOURCE = os.path.join(ROOT, "paper_2609_33762_amd", "csrc", "ea_copy_kernels.hip")
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "piece_copy_qwen3_turn_hbm_bytes.md")
TRACE_SUMMARY = os.path.join(ROOT, "profiles", "piece_copy_qwen3_turn_kernel_trace.md")
PLANS_SUMMARY = os.path.join(ROOT, "profiles", "transfer_plans_size_classes.md")
N_ISO = {"store": 5, "load": 5, "gather": 20, "scatter": 20}


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def kernel_source_hash():
    return hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest()[:16]


_STREAMS = []


def copy_streams(torch):
    """The process's two copy streams (stores, loads), created once and after
    the process has first used the default stream.  The runtime places each
    stream on one of a few hardware queues; streams created before the
    default stream's first use lose part of their overlap once it is used,
    and streams created beyond the hardware queues share them (measured: the
    turn's duplex falls from 87 to 68-77 and 56 GB/s)."""
    if not _STREAMS:
        torch.zeros(1, device="cuda")  # a kernel on the default stream
        torch.cuda.synchronize()
        _STREAMS.extend([torch.cuda.Stream(), torch.cuda.Stream()])
    return _STREAMS[0], _STREAMS[1]


def event_ms(torch, fn, stream, reps, warm=1):
    """Average duration of one fn() call: `reps` back-to-back calls between
    one pair of HIP events on `stream`, after `warm` untimed calls (events
    between the calls would add their own cost to every launch).  One more
    untimed call goes onto the stream right before the start event, so the
    GPU is still busy with it while the host enqueues the first timed call:
    the interval holds the calls' GPU time and the spacing between their
    launches, not the host's latency to the first launch."""
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    fn()
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def cpu_baseline(W, n_s, n_l, prefix_tokens, refill_tokens):
    """The oracle (single thread, pinned to one core) running one full step of
    the same workload on host arrays: hash both sequences, store 2,000 pages,
    load 1,500 pages.  Cache and tier are sampled down to the pages touched."""
    import oracle
    sh = W.QWEN3
    P = n_s + n_l
    oshape = oracle.make_shape(P, sh.num_layers, sh.page_tokens, sh.num_kv_heads,
                               sh.head_dim, sh.elem_bytes)
    sz = oracle.sizes(oshape)
    cache = np.tile(W.host_bytes(W.SEED_DATA, sz["piece"]), sh.num_layers * P)
    tier = np.zeros((P, sz["slot"]), np.uint8)
    toks = np.concatenate([prefix_tokens, refill_tokens])
    offs = np.array([0, len(toks)], np.int64)  # the whole prompt, one chain
    prev = os.sched_getaffinity(0)
    os.sched_setaffinity(0, {sorted(prev)[0]})
    # a bounded sample: repeat the step until 10 s of CPU work (5 to 100 runs)
    times = {"hash": [], "store": [], "load": []}
    start = time.perf_counter()
    try:
        while len(times["hash"]) < 5 or (time.perf_counter() - start < 10.0
                                          and len(times["hash"]) < 100):
            t0 = time.perf_counter()
            oracle.hash_blocks(toks, offs, sh.page_tokens)
            t1 = time.perf_counter()
            oracle.store_blocks(oshape, cache, None, tier, np.arange(n_s, dtype=np.int32),
                                np.arange(n_l, P, dtype=np.int64))
            t2 = time.perf_counter()
            oracle.load_blocks(oshape, tier, cache, None, np.arange(n_l, 2 * n_l, dtype=np.int64),
                               np.arange(n_s, n_s + n_l, dtype=np.int32))
            t3 = time.perf_counter()
            times["hash"].append(t1 - t0)
            times["store"].append(t2 - t1)
            times["load"].append(t3 - t2)
    finally:
        os.sched_setaffinity(0, prev)
    reps = len(times["hash"])
    med = {k: float(np.median(v)) for k, v in times.items()}
    t = sum(med.values())
    moved = (n_s + n_l) * sz["page"]
    model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": round(moved / t / GB, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "hash_tokens_per_s": round(len(toks) / med["hash"], 1),
            "store_gbs": round(n_s * sz["page"] / med["store"] / GB, 3),
            "load_gbs": round(n_l * sz["page"] / med["load"] / GB, 3),
            "nproc": os.cpu_count(), "cpu_model": model,
            "sample": f"one full step (hash {len(toks)} tokens, store {n_s} pages, load {n_l} "
                      f"pages of {sz['page']} B) on a {P}-page host cache; the sum of each "
                      f"phase's median over {reps} runs",
            "ms_per_step": round(t * 1e3, 1)}


def committed_traffic():
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when it is missing or was taken on another version of the kernels."""
    if not os.path.exists(TRAFFIC_SUMMARY):
        return None
    vals, src = {}, None
    for line in open(TRAFFIC_SUMMARY):
        if line.startswith("kernel_source_sha256:"):
            src = line.split(":", 1)[1].strip()
        if line.startswith("traffic_bytes_per_launch:"):
            for kv in line.split(":", 1)[1].split():
                k, v = kv.split("=")
                vals[k] = int(v)
    if src != kernel_source_hash():
        return None
    return vals


def setup(args):
    import torch
    from paper_2609_33762_amd import api, _native as N, workloads as W
    torch.cuda.set_device(0)
    sh = W.QWEN3
    dev = torch.device("cuda", 0)
    t0 = time.perf_counter()
    kv = torch.empty(sh.cache_bytes, dtype=torch.uint8, device=dev)
    W.fill_bf16_normal(kv, W.SEED_DATA)
    cache = api.Cache(kv, sh.num_pages, sh.num_layers, sh.page_tokens, sh.num_kv_heads,
                      sh.head_dim, sh.elem_bytes)
    tier = api.Tier(cache, W.QWEN3_TIER_BYTES)
    plan = {"auto": N.EA_PLAN_AUTO, "direct": N.EA_PLAN_DIRECT, "staged": N.EA_PLAN_STAGED}
    tier.set_plan(N.EA_DIR_BOTH, plan[args.plan])
    log(f"setup: cache {sh.cache_bytes / 2**30:.2f} GiB, tier {tier.capacity} slots of "
        f"{tier.slot_bytes} B in {time.perf_counter() - t0:.1f} s")
    ctx = dict(torch=torch, api=api, N=N, W=W, sh=sh, dev=dev, kv=kv, cache=cache, tier=tier,
               page=tier.info["page_bytes"], slot=tier.slot_bytes,
               n_load=W.QWEN3_LOAD_PAGES, n_store=W.QWEN3_STORE_PAGES, r=W.rng(W.SEED_WORKLOAD))
    # pinned-copy peak of the host link (1 GiB contiguous, best of 10), taken
    # while the tier is still empty
    probe = torch.empty(2 << 30, dtype=torch.uint8, device=dev)
    ctx["peak"] = {"d2h": tier.peak_probe(probe, 1 << 30, N.EA_DIR_STORE, 10),
                   "h2d": tier.peak_probe(probe, 1 << 30, N.EA_DIR_LOAD, 10),
                   "bidir": tier.peak_probe(probe, 1 << 30, N.EA_DIR_BOTH, 10)}
    del probe
    log(f"pinned-copy peak GB/s: { {k: round(v, 2) for k, v in ctx['peak'].items()} }")
    # the cached prefix of the turn is already in the tier
    b = sh.page_tokens
    ctx["prefix"] = W.tokens(W.SEED_TOKENS, ctx["n_load"] * b)
    pkeys, _ = api.hash_blocks(ctx["prefix"], np.array([0, len(ctx["prefix"])]), b)
    prefix_pages = W.distinct(ctx["r"], sh.num_pages, ctx["n_load"])
    cnt, pslots = tier.alloc(pkeys)
    assert cnt == ctx["n_load"]
    tier.store(cache, prefix_pages, pslots)
    tier.unpin(pslots)
    torch.cuda.synchronize()
    ctx["pslots"] = pslots
    return ctx


def run_steps(ctx, args):
    torch, api, W, sh, tier, cache = (ctx[k] for k in ("torch", "api", "W", "sh", "tier", "cache"))
    n_load, n_store, r, b = ctx["n_load"], ctx["n_store"], ctx["r"], sh.page_tokens
    policy = api.make_policy(kappa=256, block_tokens=b,
                             beta_rank=sh.num_layers * sh.piece_bytes // b)
    total = args.warmup + args.steps
    refills = [W.tokens(W.SEED_TOKENS + 100 + k, n_store * b) for k in range(total)]
    store_pages, load_dst = [], []
    for k in range(total):
        sp = W.distinct(r, sh.num_pages, n_store)
        store_pages.append(sp)
        load_dst.append(W.distinct(r, sh.num_pages, n_load, exclude=sp))
    # each step's prompt is the cached prefix followed by a fresh refill; its
    # keys form one chain over the whole prompt (the refill's keys depend on
    # the prefix), computed at the request's first lookup
    seqs = [np.concatenate([ctx["prefix"], refills[k]]) for k in range(total)]
    offs = np.array([0, (n_load + n_store) * b], np.int64)
    s_store, s_load = copy_streams(torch)
    ev = {k: [] for k in ("s0", "s1", "l0", "l1")}

    def step(k, timed):
        keys, _ = api.hash_blocks(seqs[k], offs, b)
        h, hslots = tier.lookup(keys)  # stops at the refill's first block
        assert h == n_load, h
        if timed:
            ev["l0"].append(torch.cuda.Event(enable_timing=True))
            ev["l0"][-1].record(s_load)
        tier.load(cache, hslots, load_dst[k], stream=s_load)
        if timed:
            ev["l1"].append(torch.cuda.Event(enable_timing=True))
            ev["l1"][-1].record(s_load)
        # the write rule over the whole request (n tokens, h of them hit);
        # deduplication leaves the prefix's blocks out of the mask
        _, mask = tier.admission(policy, len(seqs[k]), h * b, 1, k, keys)
        _, slots = tier.alloc(keys, mask)
        slots = slots[n_load:]
        ok = slots >= 0
        if timed:
            ev["s0"].append(torch.cuda.Event(enable_timing=True))
            ev["s0"][-1].record(s_store)
        tier.store(cache, store_pages[k][ok], slots[ok], stream=s_store)
        if timed:
            ev["s1"].append(torch.cuda.Event(enable_timing=True))
            ev["s1"][-1].record(s_store)
        tier.unpin(slots[ok])
        tier.unpin(hslots)
        return int(ok.sum())

    for k in range(args.warmup):
        step(k, False)
    torch.cuda.synchronize()
    stored = []
    t0 = time.perf_counter()
    for k in range(args.warmup, total):
        stored.append(step(k, True))
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    store_ms = [a.elapsed_time(c) for a, c in zip(ev["s0"], ev["s1"])]
    load_ms = [a.elapsed_time(c) for a, c in zip(ev["l0"], ev["l1"])]
    page = ctx["page"]
    res = {"ms": elapsed / args.steps * 1e3,
           "gbs": (sum(stored) + args.steps * n_load) * page / elapsed / GB,
           "store_ms": float(np.mean(store_ms)), "load_ms": float(np.mean(load_ms)),
           # each timed store is one kernel launch of `stored` pages, each load
           # one launch of n_load pages; HIP events on the launching stream
           "store_gbs_in_step": sum(stored) * page / (sum(store_ms) * 1e-3) / GB,
           "load_gbs_in_step": args.steps * n_load * page / (sum(load_ms) * 1e-3) / GB,
           "stored_pages": stored, "tier": tier.stats()}
    ctx["last_store_pages"], ctx["last_load_dst"], ctx["last_refill"] = (
        store_pages[-1], load_dst[-1], refills[-1])
    log(f"step {res['ms']:.2f} ms, {res['gbs']:.1f} GB/s over the link; in-step store "
        f"{res['store_ms']:.2f} ms ({res['store_gbs_in_step']:.1f} GB/s), load "
        f"{res['load_ms']:.2f} ms ({res['load_gbs_in_step']:.1f} GB/s); evictions "
        f"{res['tier']['evictions_total']}")
    return res


def isolated(ctx):
    """Each direction alone (2,000 pages stored to the consecutive slots a
    fresh allocation hands out, the 1,500-page prefix loaded from its slots),
    the same with random slots, and the HBM gather/scatter kernels; ends with
    a plain 1 GiB device copy that calibrates the HBM byte counters."""
    torch, W, sh, tier, cache, dev = (ctx[k] for k in ("torch", "W", "sh", "tier", "cache", "dev"))
    n_store, n_load, page, slot, r = ctx["n_store"], ctx["n_load"], ctx["page"], ctx["slot"], ctx["r"]
    sp = ctx.get("last_store_pages")
    if sp is None:
        sp = W.distinct(r, sh.num_pages, n_store)
    dst = ctx.get("last_load_dst")
    if dst is None:
        dst = W.distinct(r, sh.num_pages, n_load, exclude=sp)
    cur = torch.cuda.current_stream()
    torch.cuda.synchronize()
    # raw stores: from here on the tier's contents no longer matter
    # random slots first, so that the last launches of each kernel are the
    # consecutive-slot ones the profile summaries pick out
    out = {}
    rnd = W.distinct(r, tier.capacity, n_store)
    out["store_rnd_ms"] = event_ms(torch, lambda: tier.store(cache, sp, rnd, stream=cur), cur, 3)
    out["load_rnd_ms"] = event_ms(torch, lambda: tier.load(cache, rnd[:n_load], dst, stream=cur),
                                  cur, 3)
    slots = np.arange(n_store, dtype=np.int64)
    out["store_ms"] = event_ms(torch, lambda: tier.store(cache, sp, slots, stream=cur), cur,
                               N_ISO["store"])
    out["load_ms"] = event_ms(torch, lambda: tier.load(cache, ctx["pslots"], dst, stream=cur), cur,
                              N_ISO["load"])
    staging = torch.empty(n_store * slot, dtype=torch.uint8, device=dev)
    out["gather_ms"] = event_ms(torch, lambda: cache.gather(sp, staging, stream=cur), cur,
                                N_ISO["gather"])
    out["scatter_ms"] = event_ms(torch, lambda: cache.scatter(staging, sp, stream=cur), cur,
                                 N_ISO["scatter"])
    calib = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    calib.copy_(staging[: 1 << 30])
    torch.cuda.synchronize()
    del staging, calib
    out["store_gbs"] = n_store * page / (out["store_ms"] * 1e-3) / GB
    out["load_gbs"] = n_load * page / (out["load_ms"] * 1e-3) / GB
    out["store_rnd_gbs"] = n_store * page / (out["store_rnd_ms"] * 1e-3) / GB
    out["load_rnd_gbs"] = n_load * page / (out["load_rnd_ms"] * 1e-3) / GB
    out["gather_gbs"] = 2 * n_store * slot / (out["gather_ms"] * 1e-3) / GB
    out["scatter_gbs"] = 2 * n_store * slot / (out["scatter_ms"] * 1e-3) / GB
    pk = ctx["peak"]
    log(f"alone: store {out['store_gbs']:.1f} GB/s ({out['store_gbs'] / pk['d2h']:.1%} of pinned "
        f"D2H), load {out['load_gbs']:.1f} GB/s ({out['load_gbs'] / pk['h2d']:.1%} of pinned H2D); "
        f"random slots {out['store_rnd_gbs']:.1f} / {out['load_rnd_gbs']:.1f}; HBM gather "
        f"{out['gather_gbs']:.0f} GB/s, scatter {out['scatter_gbs']:.0f} GB/s")
    return out


# ------------------------------------------------- the other workloads

def _line(workload, value, unit, ms, steps, extra, higher=True):
    return {"metric": "host-link GB/s for KV block store/load; HBM GB/s of paged gather/scatter",
            "value": value, "unit": unit, "n_gpus": 1, "steps": steps, "warmup": 0,
            "ms_per_step": ms, "higher_is_better": higher, "scaling": "weak",
            "vs_baseline": None, "dtype": "u8", "data": "synthetic",
            "config": {"workload": workload}, **extra}


def _pinned_one_core(fn):
    """Run fn() on one core (the first of this process's), then restore."""
    prev = os.sched_getaffinity(0)
    os.sched_setaffinity(0, {sorted(prev)[0]})
    try:
        return fn()
    finally:
        os.sched_setaffinity(0, prev)


def _pool_cpu_baseline(records, sh, chunk_pages, tier_bytes, kappa, window, mode=0):
    """The oracle on one core replays every turn's metadata (lookup, write
    rule, allocation, store marks, unpins) from the run's records and checks
    each result against the library's; then it times host copies of 256
    slots each way at the pool's slot size."""
    import oracle
    C = chunk_pages
    b = sh.page_tokens * C
    beta = sh.num_layers * sh.piece_bytes // sh.page_tokens
    oshape = oracle.make_shape(sh.num_pages, sh.num_layers, sh.page_tokens, sh.num_kv_heads,
                               sh.head_dim, sh.elem_bytes, chunk_pages=C)
    opol = oracle.make_policy(kappa=kappa, block_tokens=b, beta=beta, activity_window=window,
                              mode=mode)

    def replay():
        ot = oracle.Tier(oshape, tier_bytes)
        ok = True
        t0 = time.perf_counter()
        for rec in records:
            h, hs = ot.lookup(rec.keys)
            ok &= bool(h == rec.hit and np.array_equal(hs, rec.hit_slots))
            save, mask = ot.admission(opol, rec.n_tokens, rec.hit * b, rec.agent, rec.turn,
                                      rec.keys)
            ok &= bool(save == rec.save and np.array_equal(mask, rec.mask))
            _, slots = ot.alloc(rec.keys, mask)
            ok &= bool(np.array_equal(slots, rec.alloc_slots))
            good = slots >= 0
            ot.mark_stored(slots[good])
            if good.any():
                ot.unpin(slots[good])
            if h:
                ot.unpin(hs)
        return ok, time.perf_counter() - t0

    ok, replay_s = _pinned_one_core(replay)
    # copies: 256 pages (in slots of C pages) stored from and loaded back
    # into a host cache of those pages
    n = max(1, 256 // C)
    mini = oracle.make_shape(n * C, sh.num_layers, sh.page_tokens, sh.num_kv_heads, sh.head_dim,
                             sh.elem_bytes, chunk_pages=C)
    sz = oracle.sizes(mini)
    cache = np.tile(W_host_bytes(sz["piece"]), sh.num_layers * n * C)
    otier = np.zeros((n, sz["slot"]), np.uint8)
    ids = np.arange(n * C, dtype=np.int32)
    sl = np.arange(n, dtype=np.int64)

    def copies():
        ts, tl = [], []
        for _ in range(5):
            t0 = time.perf_counter()
            oracle.store_blocks(mini, cache, None, otier, ids, sl)
            t1 = time.perf_counter()
            oracle.load_blocks(mini, otier, cache, None, sl, ids)
            tl.append(time.perf_counter() - t1)
            ts.append(t1 - t0)
        return float(np.median(ts)), float(np.median(tl))

    t_s, t_l = _pinned_one_core(copies)
    moved = n * sz["slot"]
    return {"value": round(2 * moved / (t_s + t_l) / GB, 3), "unit": "GB/s", "cores": 1,
            "kind": "oracle", "store_gbs": round(moved / t_s / GB, 3),
            "load_gbs": round(moved / t_l / GB, 3),
            "metadata_replay_s": round(replay_s, 3), "turns_replayed": len(records),
            "oracle_replay_ok": ok,
            "sample": f"metadata of all {len(records)} turns replayed on the oracle's tier; "
                      f"copies of {n} slots of {sz['slot']} B each way, median of 5"}


def W_host_bytes(n):
    from paper_2609_33762_amd import workloads as W
    return W.host_bytes(W.SEED_DATA, n)


def run_agent_pool(args):
    """64 agents round-robin, 24 turns each (1,536 turns), 64 GiB tier."""
    import torch
    from paper_2609_33762_amd import api, drivers, workloads as W
    torch.cuda.set_device(0)
    sh = W.QWEN3
    kv = torch.empty(sh.cache_bytes, dtype=torch.uint8, device="cuda")
    cache = api.Cache(kv, sh.num_pages, sh.num_layers, sh.page_tokens, sh.num_kv_heads,
                      sh.head_dim, sh.elem_bytes)
    tier = api.Tier(cache, W.POOL_TIER_BYTES)
    beta = sh.num_layers * sh.piece_bytes // sh.page_tokens
    pol = api.make_policy(kappa=256, block_tokens=sh.page_tokens, beta_rank=beta,
                          activity_window=W.POOL_AGENTS)
    # loads and stores on their own streams: a turn's store overlaps the next
    # turn's load on the host link
    s_store, s_load = copy_streams(torch)
    pool = drivers.AgentPool(torch, cache, tier, kv, sh, pol, verify=False, time_fill=True,
                             load_stream=s_load, store_stream=s_store)
    turns = args.turns_per_agent * W.POOL_AGENTS
    hits = declined = stored = 0
    gamma = []
    records = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(turns):
        rec = pool.turn()
        records.append(rec)
        hits += rec.hit
        declined += int(not rec.save)
        stored += rec.stored
        if t % W.POOL_AGENTS == W.POOL_AGENTS - 1:
            st = tier.stats()
            gamma.append(round(st["working_set"] / W.POOL_TIER_BYTES, 3))
    torch.cuda.synchronize()
    # the synthetic KV fill stands in for prefill compute: not part of the path
    el = time.perf_counter() - t0 - pool.fill_seconds
    st = tier.stats()
    moved = pool.bytes_loaded + pool.bytes_stored
    extra = {"pool": {"turns": turns, "fill_seconds_excluded": round(pool.fill_seconds, 3),
                      "hit_blocks": hits, "stored_blocks": stored,
                      "declined_requests": declined, "evictions": st["evictions_total"],
                      "gamma_H_per_round": gamma, "bytes_loaded": pool.bytes_loaded,
                      "bytes_stored": pool.bytes_stored}}
    extra["pool"]["reference_model"] = drivers.stack_report(
        records, tier.capacity, tier.slot_bytes, [16 << 30, 32 << 30, 64 << 30, 128 << 30,
                                                  256 << 30])
    extra["pool"]["reference_model"].pop("hits_tier_order_per_request")
    log(f"reference model: {extra['pool']['reference_model']}")
    tier.close()
    cache.close()
    if not args.no_cpu_baseline:
        extra["cpu_baseline"] = _pool_cpu_baseline(records, sh, 1, W.POOL_TIER_BYTES, 256,
                                                   W.POOL_AGENTS)
        log(f"cpu baseline: {extra['cpu_baseline']}")
    return _line("agent_pool: 64 agents x %d turns, contexts 8k->64k, 64 GiB tier"
                 % args.turns_per_agent, round(moved / el / GB, 3), "GB/s",
                 round(el / turns * 1e3, 3), turns, extra)


def run_agent_pool_chunked(args):
    """The agent pool at the paper's deployment parameters on one TP8 rank:
    24 KiB per token, 1,024-token host chunks (64 pages, 24 MiB), 16 agents,
    kappa = 8 chunks, host tiers of 5, 10 and 40 GiB (213, 426 and 1,706
    chunks), 24 turns per agent; loads and stores on two streams.  Each tier
    runs under the three admission modes of section 4: offload without
    admission (p = 0), fixed admission (p = 1) and the conditioned rule."""
    import torch
    from paper_2609_33762_amd import api, drivers, workloads as W
    torch.cuda.set_device(0)
    sh, C = W.QWEN3_TP8, W.CHUNK_PAGES
    kv = torch.empty(sh.cache_bytes, dtype=torch.uint8, device="cuda")
    cache = api.Cache(kv, sh.num_pages, sh.num_layers, sh.page_tokens, sh.num_kv_heads,
                      sh.head_dim, sh.elem_bytes)
    beta = sh.num_layers * sh.piece_bytes // sh.page_tokens
    agents = 16
    turns = args.turns_per_agent * agents
    from paper_2609_33762_amd import _native as N
    modes = {"offload": N.EA_ADMIT_ALWAYS, "fixed": N.EA_ADMIT_FIXED,
             "conditioned": N.EA_ADMIT_CONDITIONED}
    runs, total_moved, total_s = {}, 0, 0.0
    for gib, (mname, mode) in [(g, m) for g in (5, 10, 40) for m in modes.items()]:
        tier = api.Tier(cache, gib << 30, chunk_pages=C)
        pol = api.make_policy(kappa=8, block_tokens=C * sh.page_tokens, beta_rank=beta,
                              activity_window=agents, mode=mode)
        s_store, s_load = copy_streams(torch)
        pool = drivers.AgentPool(torch, cache, tier, kv, sh, pol, agents=agents, verify=False,
                                 time_fill=True, load_stream=s_load, store_stream=s_store)
        records = []
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(turns):
            records.append(pool.turn())
        torch.cuda.synchronize()
        el = time.perf_counter() - t0 - pool.fill_seconds
        st = tier.stats()
        moved = pool.bytes_loaded + pool.bytes_stored
        total_moved += moved
        total_s += el
        rep = drivers.stack_report(records, tier.capacity, tier.slot_bytes)
        rep.pop("hits_tier_order_per_request")
        replay = None
        if not args.no_cpu_baseline:
            replay = _pool_cpu_baseline(records, sh, C, gib << 30, 8, agents, mode)
        runs[f"{gib}GiB_{mname}"] = {
            "K_H": tier.capacity, "gbs": round(moved / el / GB, 2),
            "ms_per_turn": round(el / turns * 1e3, 3),
            "hit_chunks": int(sum(r.hit for r in records)),
            "prompt_chunks": int(sum(len(r.keys) for r in records)),
            "stored_chunks": int(sum(r.stored for r in records)),
            "declined_requests": int(sum(not r.save for r in records)),
            "evictions": st["evictions_total"], "reference_model": rep,
            "oracle_replay_ok": None if replay is None else replay["oracle_replay_ok"],
            "oracle_metadata_replay_s": None if replay is None else replay["metadata_replay_s"]}
        r = runs[f"{gib}GiB_{mname}"]
        log(f"chunked pool {gib} GiB {mname}: hit {r['hit_chunks']} of {r['prompt_chunks']}, "
            f"stored {r['stored_chunks']}, declined {r['declined_requests']}, evictions "
            f"{r['evictions']}, {r['gbs']} GB/s, declined meeting Prop. 1 "
            f"{rep['declined_meeting_condition']}, tier-order model {rep['hits_model_tier_order']}")
        tier.close()
    cache.close()
    extra = {"pool_chunked": runs}
    if not args.no_cpu_baseline:
        extra["cpu_baseline"] = dict(replay, oracle_replay_ok=all(
            r["oracle_replay_ok"] for r in runs.values()))
        extra["cpu_baseline"]["sample"] = ("metadata of every turn of all nine runs replayed on "
                                           "the oracle's tier (replay time of the last run); "
                                           + replay["sample"].split("; ", 1)[1])
    return _line("agent_pool_chunked: one TP8 rank, 1,024-token chunks, 16 agents x %d turns, "
                 "5/10/40 GiB tiers x 3 admission modes" % args.turns_per_agent,
                 round(total_moved / total_s / GB, 3), "GB/s",
                 round(total_s / (9 * turns) * 1e3, 3), 9 * turns, extra)


def _dense_cpu_baseline(sh, calls=2000):
    """The oracle on one core: `calls` alternating store / load calls of 1-8
    random non-adjacent pages between a 256-page host cache and a 256-slot
    host tier of the dense shape (2 MiB pages); per-call time."""
    import oracle
    from paper_2609_33762_amd import drivers, workloads as W
    n_pages = 256
    o = oracle.make_shape(n_pages, sh.num_layers, sh.page_tokens, sh.num_kv_heads, sh.head_dim,
                          sh.elem_bytes)
    sz = oracle.sizes(o)
    cache = np.tile(W.host_bytes(W.SEED_DATA, sz["piece"]), sh.num_layers * n_pages)
    otier = np.zeros((n_pages, sz["slot"]), np.uint8)
    r = W.rng(W.SEED_WORKLOAD)
    plan = []
    for i in range(calls):
        k = int(r.integers(1, 9))
        plan.append((i % 2, drivers.non_adjacent_pages(r, n_pages, k).astype(np.int32),
                     r.choice(n_pages, size=k, replace=False).astype(np.int64)))

    def run():
        ts, moved = [], 0
        for op, pages, slots in plan:
            t0 = time.perf_counter()
            if op == 0:
                oracle.store_blocks(o, cache, None, otier, pages, slots)
            else:
                oracle.load_blocks(o, otier, cache, None, slots, pages)
            ts.append(time.perf_counter() - t0)
            moved += len(pages) * sz["page"]
        return np.array(ts), moved

    ts, moved = _pinned_one_core(run)
    return {"value": round(moved / ts.sum() / GB, 3), "unit": "GB/s", "cores": 1,
            "kind": "oracle", "per_call_ms_p50": round(float(np.percentile(ts, 50)) * 1e3, 4),
            "per_call_ms_p99": round(float(np.percentile(ts, 99)) * 1e3, 4),
            "sample": f"{calls} alternating store/load calls of 1-8 pages of {sz['page']} B on "
                      f"a {n_pages}-page host cache and tier"}


def run_dense_scattered(args):
    """10,000 alternating store/load calls of 1-8 non-adjacent 2 MiB pages."""
    import torch
    from paper_2609_33762_amd import api, drivers, workloads as W
    torch.cuda.set_device(0)
    sh = W.DENSE
    kv = torch.empty(sh.cache_bytes, dtype=torch.uint8, device="cuda")
    W.fill_bf16_normal(kv, W.SEED_DATA)
    cache = api.Cache(kv, sh.num_pages, sh.num_layers, sh.page_tokens, sh.num_kv_heads,
                      sh.head_dim, sh.elem_bytes)
    tier = api.Tier(cache, W.DENSE_TIER_SLOTS * sh.num_layers * sh.piece_bytes)
    page = tier.info["page_bytes"]
    # per-call latency: enqueue to completion, one call at a time
    drv = drivers.DenseScattered(cache, tier, sh)
    lat, moved = [], 0
    for i in range(W.DENSE_CALLS):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        _, pages, _ = drv.call(i)
        torch.cuda.synchronize()
        lat.append(time.perf_counter() - t0)
        moved += len(pages) * page
    lat_ms = np.array(lat) * 1e3
    # throughput: the same calls issued back to back
    drv2 = drivers.DenseScattered(cache, tier, sh, seed=W.SEED_WORKLOAD + 1)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    moved2 = 0
    for i in range(W.DENSE_CALLS):
        _, pages, _ = drv2.call(i)
        moved2 += len(pages) * page
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    extra = {"latency_ms": {"p50": round(float(np.percentile(lat_ms, 50)), 4),
                            "p99": round(float(np.percentile(lat_ms, 99)), 4),
                            "mean_bytes_per_call": moved / W.DENSE_CALLS,
                            "serial_gbs": round(moved / lat_ms.sum() * 1e3 / GB, 3)},
             "calls_per_s": round(W.DENSE_CALLS / el, 1)}
    tier.close()
    cache.close()
    if not args.no_cpu_baseline:
        extra["cpu_baseline"] = _dense_cpu_baseline(sh)
        log(f"cpu baseline: {extra['cpu_baseline']}")
    return _line("dense_scattered: 32 layers x 8 heads x d128 bf16, 10,000 calls of 1-8 pages",
                 round(moved2 / el / GB, 3), "GB/s", round(el / W.DENSE_CALLS * 1e3, 4),
                 W.DENSE_CALLS, extra)


def _layered_once(torch, api, W, sh, steps, cpu=True):
    """Load the 4,096-page prefix of shape sh one layer at a time, `steps`
    timed repetitions after one untimed; a consumer stream waits on each
    layer's event and checksums that layer of every destination page (the
    stand-in for attention over the layer).  Returns the bench figures, with
    the oracle's check of the consumer's checksums and its timing."""
    L, P = sh.num_layers, sh.num_pages
    kv = torch.empty(sh.cache_bytes, dtype=torch.uint8, device="cuda")
    W.fill_random_bytes(kv, W.SEED_DATA)
    sc = torch.empty(L * P * 8, dtype=torch.uint8, device="cuda")
    W.fill_random_bytes(sc, W.SEED_DATA + 1)
    cache = api.Cache(kv, P, L, sh.page_tokens, sh.num_kv_heads, sh.head_dim, sh.elem_bytes,
                      scales=sc)
    n = W.LAYERED_PREFIX_PAGES
    tier = api.Tier(cache, n * (L * sh.piece_bytes + 512))
    r = W.rng(W.SEED_IDS)
    src = W.distinct(r, P, n)
    dst = np.setdiff1d(np.arange(P), src)
    tier.store(cache, src, np.arange(n))
    cons_s, copy_s = copy_streams(torch)
    sums = torch.zeros((L, n), dtype=torch.int64, device="cuda")
    res, cons = [], []
    for rep in range(steps + 1):
        start = torch.cuda.Event(enable_timing=True)
        events = [torch.cuda.Event(enable_timing=True) for _ in range(L)]
        done = [torch.cuda.Event(enable_timing=True) for _ in range(L)]
        torch.cuda.synchronize()
        start.record(copy_s)
        tier.load_layered(cache, np.arange(n), dst, copy_s, events)
        for l in range(L):
            cons_s.wait_event(events[l])
            cache.layer_checksum(l, dst, sums[l], stream=cons_s)
            done[l].record(cons_s)
        torch.cuda.synchronize()
        if rep:
            res.append([start.elapsed_time(e) for e in events])
            cons.append([start.elapsed_time(e) for e in done])
    res, cons = np.array(res), np.array(cons)
    total_ms = float(np.median(res[:, -1]))
    moved = n * tier.slot_bytes
    out = {"gbs": round(moved / (total_ms * 1e-3) / GB, 3), "ms": round(total_ms, 3),
           "slot_bytes": tier.slot_bytes,
           "time_to_first_layer_ms": round(float(np.median(res[:, 0])), 4),
           "per_layer_ms": round(float(np.median(np.diff(res, axis=1))), 4),
           "layer_done_ms": [round(float(x), 3) for x in np.median(res, axis=0)],
           "consumer": {
               "kernel": "ea_layer_checksum: XOR of each destination page's layer piece",
               "done_ms": [round(float(x), 3) for x in np.median(cons, axis=0)],
               "finish_after_last_layer_ms": round(float(np.median(cons[:, -1] - res[:, -1])), 4),
               "lag_per_layer_ms": round(float(np.median(cons - res)), 4),
               "layers_consumed_before_load_done": int(np.median((cons < res[:, -1:]).sum(1)))}}
    if cpu:
        out["cpu_baseline"] = _layered_cpu_baseline(sh, tier, dst, sums.cpu().numpy())
    tier.close()
    cache.close()
    del kv, sc
    return out


def _layered_cpu_baseline(sh, tier, dst, sums):
    """The oracle on one core: the layer-by-layer load of the tier's image
    into a host cache of the destination pages, then each layer's checksum
    (compared with the consumer's), timed per layer."""
    import oracle
    n, L = len(dst), sh.num_layers
    o = oracle.make_shape(n, L, sh.page_tokens, sh.num_kv_heads, sh.head_dim, sh.elem_bytes,
                          True)
    host = tier.host_view()
    ocache = np.zeros(L * n * sh.piece_bytes, np.uint8)
    osc = np.zeros(L * n * 8, np.uint8)
    idx = np.arange(n, dtype=np.int32)
    prev = os.sched_getaffinity(0)
    os.sched_setaffinity(0, {sorted(prev)[0]})
    t_load, t_sum, ok = [], [], True
    try:
        for l in range(L):
            t0 = time.perf_counter()
            oracle.load_layer(o, host, ocache, osc, np.arange(n, dtype=np.int64), idx, l)
            t1 = time.perf_counter()
            want = oracle.layer_checksum(o, ocache, osc, l, idx)
            t2 = time.perf_counter()
            t_load.append(t1 - t0)
            t_sum.append(t2 - t1)
            ok &= bool(np.array_equal(sums[l].view(np.uint64), want))
    finally:
        os.sched_setaffinity(0, prev)
    moved = n * tier.slot_bytes
    return {"value": round(moved / sum(t_load) / GB, 3), "unit": "GB/s", "cores": 1,
            "kind": "oracle", "layer_checksum_ms": round(float(np.median(t_sum)) * 1e3, 2),
            "load_layer_ms": round(float(np.median(t_load)) * 1e3, 2),
            "consumer_checksums_match_oracle": ok,
            "sample": f"the whole prefix: {L} layers of {n} pages, each loaded from the tier "
                      f"image and checksummed"}


def run_layered(args):
    """64k-token fp8 prefix (4,096 pages, 48 layers, per-page scales) loaded
    one layer at a time, each layer signalled by an event; then the same
    prefix on one TP8 rank's share (1 KV head, 4 KiB pieces)."""
    import torch
    from paper_2609_33762_amd import api, workloads as W
    torch.cuda.set_device(0)
    full = _layered_once(torch, api, W, W.LAYERED, args.steps)
    log(f"layered 4 heads: {full['gbs']} GB/s, {full['per_layer_ms']} ms per layer")
    torch.cuda.empty_cache()
    shard = _layered_once(torch, api, W, W.LAYERED_TP8, args.steps, cpu=False)
    log(f"layered 1 head (TP8 shard): {shard['gbs']} GB/s, {shard['per_layer_ms']} ms per layer")
    cpu = full.pop("cpu_baseline")
    extra = {"layered": {k: v for k, v in full.items() if k not in ("gbs", "ms")},
             "tp8_shard": shard, "cpu_baseline": cpu}
    return _line("layered_fp8: 64k-token prefix, 48 layers x 4 heads x d128 fp8 + scales",
                 full["gbs"], "GB/s", full["ms"], args.steps, extra)


def run_tiny(args):
    """The tiny case: store 32 pages, load them into 32 other pages, hash
    4 x 512 tokens.  Launch-bound by construction (512 KiB per op)."""
    import torch
    from paper_2609_33762_amd import api, workloads as W
    torch.cuda.set_device(0)
    sh = W.TINY
    kv = torch.empty(sh.cache_bytes, dtype=torch.uint8, device="cuda")
    W.fill_bf16_normal(kv, W.SEED_DATA)
    cache = api.Cache(kv, sh.num_pages, sh.num_layers, sh.page_tokens, sh.num_kv_heads,
                      sh.head_dim, sh.elem_bytes)
    tier = api.Tier(cache, W.TINY_TIER_SLOTS * sh.num_layers * sh.piece_bytes)
    r = W.rng(W.SEED_IDS)
    src = W.distinct(r, sh.num_pages, 32)
    dst = W.distinct(r, sh.num_pages, 32, exclude=src)
    slots = W.distinct(r, tier.capacity, 32)
    toks, offs = W.sequences(W.SEED_TOKENS, [512] * 4)
    steps = max(args.steps, 50)
    for _ in range(5):
        api.hash_blocks(toks, offs, sh.page_tokens)
        tier.store(cache, src, slots)
        tier.load(cache, slots, dst)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        api.hash_blocks(toks, offs, sh.page_tokens)
        tier.store(cache, src, slots)
        tier.load(cache, slots, dst)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    moved = 2 * 32 * tier.info["page_bytes"] * steps
    tier.close()
    cache.close()
    extra = {}
    if not args.no_cpu_baseline:
        extra["cpu_baseline"] = _tiny_cpu_baseline(sh, W, src, dst, slots, toks, offs)
        log(f"cpu baseline: {extra['cpu_baseline']}")
    return _line("tiny: 2 layers x 2 heads x d64 bf16, 32 pages stored and loaded, 4 x 512 "
                 "tokens hashed", round(moved / el / GB, 3), "GB/s", round(el / steps * 1e3, 4),
                 steps, extra)


def _tiny_cpu_baseline(sh, W, src, dst, slots, toks, offs):
    """The oracle on one core running the tiny step on host arrays (hash
    4 x 512 tokens, store 32 pages, load them into 32 others), repeated for
    about two seconds; medians per phase."""
    import oracle
    o = oracle.make_shape(sh.num_pages, sh.num_layers, sh.page_tokens, sh.num_kv_heads,
                          sh.head_dim, sh.elem_bytes)
    sz = oracle.sizes(o)
    cache = np.tile(W.host_bytes(W.SEED_DATA, sz["piece"]), sh.num_layers * sh.num_pages)
    otier = np.zeros((W.TINY_TIER_SLOTS, sz["slot"]), np.uint8)

    def run():
        t = {"hash": [], "store": [], "load": []}
        end = time.perf_counter() + 2.0
        while time.perf_counter() < end or len(t["hash"]) < 5:
            t0 = time.perf_counter()
            oracle.hash_blocks(toks, offs, sh.page_tokens)
            t1 = time.perf_counter()
            oracle.store_blocks(o, cache, None, otier, src, slots)
            t2 = time.perf_counter()
            oracle.load_blocks(o, otier, cache, None, slots, dst)
            t3 = time.perf_counter()
            t["hash"].append(t1 - t0)
            t["store"].append(t2 - t1)
            t["load"].append(t3 - t2)
        return {k: float(np.median(v)) for k, v in t.items()}, len(t["hash"])

    med, reps = _pinned_one_core(run)
    moved = 2 * 32 * sz["page"]
    step = sum(med.values())
    return {"value": round(moved / step / GB, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "ms_per_step": round(step * 1e3, 4),
            "hash_tokens_per_s": round(int(offs[-1]) / med["hash"], 1),
            "sample": f"the tiny step on host arrays, medians over {reps} runs"}


# ------------------------------------------------------------ profiles

def _short(name):
    for key, short in (("copy_host_link<0", "store"), ("copy_host_link<1", "load"),
                       ("copy_hbm<0", "gather"), ("copy_hbm<1", "scatter"),
                       ("copy_hbm_args<0", "gather"), ("copy_hbm_args<1", "scatter"),
                       ("sha256_chain_lane", "sha256_chain_lane"),
                       ("sha256_chain_split", "sha256_chain_split"),
                       ("sha256_chain", "sha256_chain"), ("sha256_midstates", "sha256_midstates"),
                       ("copyBuffer", "rocclr_copyBuffer")):
        if key in name:
            return short
    return None


SIDE_WORKLOADS = ("layered_fp8", "dense_scattered", "tp8_shard", "load_cost", "agent_pool",
                  "agent_pool_chunked")
WORKLOADS_SUMMARY = os.path.join(ROOT, "profiles", "side_workloads_kernel_trace.md")


def summarize_workloads(d):
    """Write the kernel-trace summary of the side workloads from directory d:
    for each workload w, d/w.json (its bench line) and d/w/w_kernel_trace.csv
    (rocprofv3 --kernel-trace --output-format csv of that bench run)."""
    cmd = ("rocprofv3 --kernel-trace --stats --output-format csv -d bench_out/prof_wl/{w} -o {w} "
           "-- python3 bench.py --workload {w} --detail bench_out/prof_wl/{w}/detail.json "
           "> bench_out/prof_wl/{w}.json")
    lines = ["# Kernel durations of the side workloads (kernel traces)", "",
             "Commands (from the repository root on the MI355X), for each workload `{w}` of "
             + ", ".join(f"`{w}`" for w in SIDE_WORKLOADS) + ":", "", "    " + cmd,
             "    python3 bench.py --summarize-workloads bench_out/prof_wl", "",
             f"kernel_source_sha256: {kernel_source_hash()}", "",
             "Each table lists the kernels of the run (library kernels by role, others by "
             "name) by launched workgroups: dispatches, median, 99th percentile, mean and "
             "total duration.  `store`/`load` are `copy_host_link` (direct plan), `gather`/"
             "`scatter` `copy_hbm`.  A host-link kernel launches its working workgroups times "
             "the XCD count over the XCDs of its direction's mask, and the workgroups that land "
             "on other XCDs return at once: 32 launched for the 8 working workgroups of a store "
             "or load, 64 for the 16 of a layer of the layered load.  Untimed set-up (filling "
             "the synthetic cache, pre-storing prefixes, the one-time XCD probe `xcd_probe`) "
             "is included.", ""]
    for w in SIDE_WORKLOADS:
        line = json.load(open(os.path.join(d, f"{w}.json")))
        groups = {}
        rows = sorted(csv.DictReader(open(os.path.join(d, w, f"{w}_kernel_trace.csv"))),
                      key=lambda x: int(x["Start_Timestamp"]))
        n_layer_loads = sum(1 for x in rows if _short(x["Kernel_Name"]) == "load")
        seen_loads = 0
        for x in rows:
            k = _short(x["Kernel_Name"]) or _plain_name(x["Kernel_Name"])
            if w == "layered_fp8" and k == "load":
                # the run loads the 4-head prefix, then the 1-head (TP8) one,
                # the same number of layer kernels each
                k = "load, 4 heads" if seen_loads < n_layer_loads // 2 else "load, 1 head"
                seen_loads += 1
            wg = int(x["Grid_Size_X"]) // max(1, int(x["Workgroup_Size_X"]))
            dur = (int(x["End_Timestamp"]) - int(x["Start_Timestamp"])) / 1e3
            groups.setdefault((k, wg), []).append(dur)
        lines += [f"## {w}", "", f"Bench line: {line['value']} {line['unit']}"
                  + (f", {line['ms_per_step']} ms per step" if line.get("ms_per_step") else "")
                  + f" ({line['config']['workload']}).", "",
                  "| kernel | workgroups | dispatches | median µs | p99 µs | mean µs | total ms |",
                  "|---|---|---|---|---|---|---|"]
        order = sorted(groups.items(), key=lambda kv: -sum(kv[1]))
        for (k, wg), v in order[:12]:
            a = np.array(v)
            lines.append(f"| {k} | {wg:,} | {len(a):,} | {np.median(a):.1f} | "
                         f"{np.percentile(a, 99):.1f} | {a.mean():.1f} | {a.sum() / 1e3:.1f} |")
        if len(order) > 12:
            rest = sum(sum(v) for _, v in order[12:])
            lines.append(f"| {len(order) - 12} other kernels | | | | | | {rest / 1e3:.1f} |")
        lines.append("")
        if w == "layered_fp8":
            from paper_2609_33762_amd import workloads as W
            n_pages = W.LAYERED_PREFIX_PAGES
            for label, shape, ev in (("4 heads", W.LAYERED, line["layered"]),
                                     ("1 head", W.LAYERED_TP8, line["tp8_shard"])):
                v = np.array([x for (k, _), vals in groups.items() if k == "load, " + label
                              for x in vals])
                piece = shape.piece_bytes
                layer_bytes = n_pages * (piece + 8)
                lines += [f"{label}: one layer's kernel moves {n_pages:,} pieces of {piece:,} B "
                          f"plus 8 B of scales each ({layer_bytes / 1e6:.2f} MB): "
                          f"{layer_bytes / (np.median(v) * 1e-6) / GB:.1f} GB/s at the median "
                          f"duration of {np.median(v):.1f} µs; the bench's event time per layer "
                          f"is {ev['per_layer_ms'] * 1e3:.1f} µs.", ""]
        if w == "dense_scattered":
            lat = line["latency_ms"]
            moved = 10000 * lat["mean_bytes_per_call"]
            ks = sum(sum(v) for (k, _), v in groups.items() if k in ("store", "load"))
            lines += [f"The run makes two series of 10,000 calls, one kernel each (one call at a "
                      f"time for the latencies, then back to back), {moved / 1e9:.1f} GB per "
                      f"series (mean {lat['mean_bytes_per_call'] / 1e6:.2f} MB per call).  Over "
                      f"the summed durations of the store and load kernels ({ks / 1e3:.1f} ms) "
                      f"that is {2 * moved / (ks * 1e-6) / GB:.1f} GB/s of kernel time, against "
                      f"{line['value']} GB/s end to end back to back and a p50 latency of "
                      f"{lat['p50'] * 1e3:.0f} µs per call from enqueue to completion.", ""]
    open(WORKLOADS_SUMMARY, "w").write("\n".join(lines))
    print(f"wrote {WORKLOADS_SUMMARY}")


def _plain_name(name):
    """A kernel's name without return type, namespaces and arguments."""
    n = name.replace("(anonymous namespace)::", "")
    n = n.split("(")[0].split("<")[0].strip()
    return n.split(" ")[-1].split("::")[-1][:48]


def summarize_profiles(d):
    """Write the committed rocprofv3 summaries from the CSVs of three runs of
    the default bench command under directory d: a kernel trace and two
    counter passes.  Store and load are read from the launches of the timed
    steps (their place in launch order is in the run's detail file), gather
    and scatter from their isolated series."""
    cmd_trace = ("rocprofv3 --kernel-trace --stats --output-format csv -d bench_out/prof_trace "
                 "-o trace -- python3 bench.py --detail bench_out/bench_detail_trace.json")
    cmd_pmc = ("rocprofv3 --pmc {c} --output-format csv -d bench_out/prof_{l} -o {l} -- python3 "
               "bench.py --no-cpu-baseline --detail bench_out/bench_detail_{l}.json")

    def pick(k, vals, plan):
        """The launches of kernel k that belong to the timed steps (store,
        load) or to the isolated series (gather, scatter)."""
        if k in plan:
            p = plan[k]
            want = p["before"] + p["timed"] + p["after"]
            if len(vals) != want:
                raise SystemExit(f"{k}: {len(vals)} launches in the profile, the run made {want}")
            return vals[p["before"]:p["before"] + p["timed"]]
        return vals[-N_ISO[k]:]

    det = json.load(open(os.path.join(d, "bench_detail_trace.json")))
    plan, steps, iso = det["dispatches"], det["steps"], det["isolated"]
    rows = list(csv.DictReader(open(os.path.join(d, "prof_trace", "trace_kernel_trace.csv"))))
    disp = {}
    for x in rows:
        k = _short(x["Kernel_Name"])
        if k:
            disp.setdefault(k, []).append((int(x["End_Timestamp"]) - int(x["Start_Timestamp"])) / 1e6)
    stats = {}
    for x in csv.DictReader(open(os.path.join(d, "prof_trace", "trace_kernel_stats.csv"))):
        k = _short(x["Name"])
        if k:
            # one row per instantiation: add calls and total time up
            c0, t0 = stats.get(k, (0, 0.0))
            stats[k] = (c0 + int(x["Calls"]), t0 + float(x["TotalDurationNs"]) / 1e6)
    stats = {k: (c, t / c) for k, (c, t) in stats.items()}
    n_store, n_load, page, slot = 2000, 1500, 1572864, 1572864
    alg = {"store": n_store * page, "load": n_load * page,
           "gather": 2 * n_store * slot, "scatter": 2 * n_store * slot}
    ev = {"store": steps["store_ms"], "load": steps["load_ms"], "gather": iso["gather_ms"],
          "scatter": iso["scatter_ms"]}
    lines = ["# Kernel durations: piece copies, Qwen3-30B-A3B turn (2,000 stored / 1,500 loaded "
             "pages of 1.5 MiB)", "",
             "Command (from the repository root on the MI355X):", "", f"    {cmd_trace}",
             "    python3 bench.py --summarize-profiles bench_out", "",
             f"kernel_source_sha256: {kernel_source_hash()}", "",
             "Store and load: the launches of the timed steps, where the two run together on "
             "two streams (launch order from the run's detail file).  Gather and scatter: their "
             "isolated series.  The HIP-event column is the same run's own timing of the same "
             "launches (events on the launching stream).", "",
             "| kernel | launches used | rocprof avg ms | HIP-event avg ms (same run) | "
             "algorithmic GB/s (rocprof) | all launches: count, --stats avg ms |",
             "|---|---|---|---|---|---|"]
    for k in ("store", "load", "gather", "scatter"):
        ds = pick(k, disp.get(k, []), plan)
        avg = float(np.mean(ds))
        c, a = stats.get(k, (0, float("nan")))
        lines.append(f"| {k} | {len(ds)} | {avg:.4f} | {ev[k]:.4f} | "
                     f"{alg[k] / (avg * 1e-3) / GB:.1f} | {c}, {a:.4f} |")
    # the hash kernels of the turn's own calls (one chain per call); the
    # line's hash block calls the same kernels afterwards
    n_turn = plan.get("hash_calls_of_turn")
    for k in ("sha256_midstates", "sha256_chain_split", "sha256_chain", "sha256_chain_lane"):
        if k in stats:
            c, a = stats[k]
            ds = disp.get(k, [])[:n_turn] if n_turn else disp.get(k, [])
            lines.append(f"| {k} | {len(ds)} | {float(np.mean(ds)):.4f} | - | - | {c}, {a:.4f} |")
    open(TRACE_SUMMARY, "w").write("\n".join(lines) + "\n")

    counters = {}
    for label, ctr in (("fetch", "FETCH_SIZE"), ("write", "WRITE_SIZE")):
        pplan = json.load(open(os.path.join(d, f"bench_detail_{label}.json")))["dispatches"]
        rows = list(csv.DictReader(open(os.path.join(d, f"prof_{label}",
                                                     f"{label}_counter_collection.csv"))))
        per = {}
        for x in rows:
            k = _short(x["Kernel_Name"])
            if k and x["Counter_Name"] == ctr:
                per.setdefault(k, []).append(float(x["Counter_Value"]))
        counters[ctr] = {k: (pick(k, v, pplan) if k in alg else v) for k, v in per.items()}
    # calibration: the last rocclr copy is the plain 1 GiB device copy
    cal_f = counters["FETCH_SIZE"]["rocclr_copyBuffer"][-1]
    cal_w = counters["WRITE_SIZE"]["rocclr_copyBuffer"][-1]
    kib = (1 << 30) / 1024
    f_fac, w_fac = kib / cal_f, kib / cal_w
    traffic = {}
    lines = ["# HBM bytes per launch: piece copies, Qwen3-30B-A3B turn", "",
             "Commands (from the repository root on the MI355X):", "",
             "    " + cmd_pmc.format(c="FETCH_SIZE", l="fetch"),
             "    " + cmd_pmc.format(c="WRITE_SIZE", l="write"),
             "    python3 bench.py --summarize-profiles bench_out", "",
             f"kernel_source_sha256: {kernel_source_hash()}", "",
             f"Calibration: a plain 1 GiB device copy (rocclr copyBuffer) reads FETCH_SIZE "
             f"{cal_f:.0f} KiB and WRITE_SIZE {cal_w:.0f} KiB for 1,048,576 KiB each way, so "
             f"FETCH_SIZE is scaled by {f_fac:.3f} and WRITE_SIZE by {w_fac:.3f}.  Reads and "
             "writes of the mapped pinned host slots count in the same counters.  Store and load "
             "are the launches of the timed steps, gather and scatter their isolated series.",
             "", "| kernel | FETCH_SIZE KiB | WRITE_SIZE KiB | scaled bytes | algorithmic bytes | "
             "ratio |", "|---|---|---|---|---|---|"]
    for k in ("store", "load", "gather", "scatter"):
        fv = counters["FETCH_SIZE"].get(k, [])
        wv = counters["WRITE_SIZE"].get(k, [])
        if not fv or not wv:
            continue
        fk, wk = float(np.mean(fv)), float(np.mean(wv))
        tb = int((fk * f_fac + wk * w_fac) * 1024)
        a2 = 2 * alg[k] if k in ("store", "load") else alg[k]
        traffic[k] = tb
        lines.append(f"| {k} | {fk:.0f} | {wk:.0f} | {tb} | {a2} | {tb / a2:.4f} |")
    lines += ["", "Algorithmic bytes count each moved byte once read and once written.", "",
              "traffic_bytes_per_launch: " + " ".join(f"{k}={v}" for k, v in traffic.items())]
    open(TRAFFIC_SUMMARY, "w").write("\n".join(lines) + "\n")
    print(open(TRACE_SUMMARY).read())
    print(open(TRAFFIC_SUMMARY).read())


HBM_COUNTER_PASSES = {
    "wr1": "TCC_EA0_WRREQ_sum TCC_EA0_WRREQ_64B_sum TCC_EA0_WRREQ_STALL_sum "
           "TCC_EA0_WRREQ_DRAM_CREDIT_STALL_sum GRBM_GUI_ACTIVE",
    "wr2": "TCC_EA0_WRREQ_LEVEL_sum TCC_TOO_MANY_EA_WRREQS_STALL_sum TCC_EA0_WRREQ_WRITE_DRAM_sum "
           "TCC_EA0_WRREQ_WRITE_GMI_32B_sum",
    "rd": "TCC_EA0_RDREQ_sum TCC_EA0_RDREQ_LEVEL_sum TCC_EA0_RDREQ_DRAM_CREDIT_STALL_sum "
          "TCC_TAG_STALL_sum",
    "tcp": "TCP_TCC_WRITE_REQ_LATENCY_sum TCP_TCC_WRITE_REQ_sum TCP_TCC_READ_REQ_LATENCY_sum "
           "TCP_TCC_READ_REQ_sum",
    "tlb": "TCP_UTCL1_TRANSLATION_MISS_sum TCP_UTCL1_TRANSLATION_HIT_sum "
           "TCP_UTCL1_STALL_UTCL2_REQ_OUT_OF_CREDITS_sum TCP_PENDING_STALL_CYCLES_sum",
}
HBM_COUNTERS_SUMMARY = os.path.join(ROOT, "profiles", "hbm_gather_scatter_counters.md")


def summarize_hbm_counters(d):
    """Write the gather-versus-scatter counter summary from directory d:
    for each unit order (entry, layer) one rocprofv3 --pmc run per pass of
    HBM_COUNTER_PASSES over `bench.py --isolated-only`; the isolated gather
    and scatter series (their last N_ISO launches) are averaged."""
    cmd = ("EA_HBM_ORDER={o} rocprofv3 --pmc {c} --output-format csv -d bench_out/hbm_{o}_{p} "
           "-o {p} -- python3 bench.py --isolated-only --no-cpu-baseline "
           "--detail bench_out/hbm_{o}_{p}.json")
    per = {}
    iso = {}
    for order in ("entry", "layer"):
        for p in HBM_COUNTER_PASSES:
            f = os.path.join(d, f"hbm_{order}_{p}", f"{p}_counter_collection.csv")
            if not os.path.exists(f):
                continue
            vals = {}
            for x in csv.DictReader(open(f)):
                k = _short(x["Kernel_Name"])
                if k in ("gather", "scatter"):
                    key = (k, x["Counter_Name"])
                    vals.setdefault(key, {}).setdefault(x.get("Dispatch_Id", len(vals)), 0.0)
                    vals[key][x.get("Dispatch_Id")] += float(x["Counter_Value"])
            for (k, c), disp in vals.items():
                v = list(disp.values())[-N_ISO[k]:]
                per[(order, k, c)] = float(np.mean(v))
            det = os.path.join(d, f"hbm_{order}_{p}.json")
            if os.path.exists(det):
                iso.setdefault(order, []).append(json.load(open(det))["isolated"])
    lines = ["# HBM gather versus scatter: what the write path does", "",
             "Qwen3-30B-A3B turn shape: 2,000 random pages of 1.5 MiB (48 pieces of 32 KiB each) "
             "gathered into a slot-layout HBM buffer and scattered back, 256 (scatter) and 512 "
             "(gather) workgroups.  Per launch averages over the isolated series "
             f"({N_ISO['gather']} launches each).", "",
             "Commands (from the repository root on the MI355X), one run per pass and order:", ""]
    for p, c in HBM_COUNTER_PASSES.items():
        lines.append("    " + cmd.format(o="entry", c=c, p=p))
    lines += ["", "and the same with EA_HBM_ORDER=layer; then "
              "`python3 bench.py --summarize-hbm-counters bench_out`.", "",
              f"kernel_source_sha256: {kernel_source_hash()}", ""]
    if iso:
        lines += ["| order | gather TB/s | scatter TB/s (HIP events, the same runs) |",
                  "|---|---|---|"]
        for o, runs in iso.items():
            g = [x["gather_gbs"] / 1e3 for x in runs]
            sc = [x["scatter_gbs"] / 1e3 for x in runs]
            lines.append(f"| {o} | {min(g):.2f}-{max(g):.2f} | {min(sc):.2f}-{max(sc):.2f} |")
        lines.append("")

    def v(o, k, c):
        return per.get((o, k, c), float("nan"))

    rows = [("EA write requests", "TCC_EA0_WRREQ_sum", None),
            ("of them 64-byte", "TCC_EA0_WRREQ_64B_sum", None),
            ("write requests to DRAM", "TCC_EA0_WRREQ_WRITE_DRAM_sum", None),
            ("32-byte writes over GMI", "TCC_EA0_WRREQ_WRITE_GMI_32B_sum", None),
            ("avg EA write latency (cycles)", "TCC_EA0_WRREQ_LEVEL_sum", "TCC_EA0_WRREQ_sum"),
            ("write stall cycles", "TCC_EA0_WRREQ_STALL_sum", None),
            ("  of them out of DRAM credits", "TCC_EA0_WRREQ_DRAM_CREDIT_STALL_sum", None),
            ("  at the pending-write limit", "TCC_TOO_MANY_EA_WRREQS_STALL_sum", None),
            ("EA read requests", "TCC_EA0_RDREQ_sum", None),
            ("avg EA read latency (cycles)", "TCC_EA0_RDREQ_LEVEL_sum", "TCC_EA0_RDREQ_sum"),
            ("read stall cycles, out of DRAM credits", "TCC_EA0_RDREQ_DRAM_CREDIT_STALL_sum", None),
            ("L2 tag stall cycles", "TCC_TAG_STALL_sum", None),
            ("avg L1-to-L2 write latency (cycles)", "TCP_TCC_WRITE_REQ_LATENCY_sum",
             "TCP_TCC_WRITE_REQ_sum"),
            ("avg L1-to-L2 read latency (cycles)", "TCP_TCC_READ_REQ_LATENCY_sum",
             "TCP_TCC_READ_REQ_sum"),
            ("address translation misses (L1 TLB)", "TCP_UTCL1_TRANSLATION_MISS_sum", None),
            ("address translation hits", "TCP_UTCL1_TRANSLATION_HIT_sum", None),
            ("stalls waiting on L2 TLB credits", "TCP_UTCL1_STALL_UTCL2_REQ_OUT_OF_CREDITS_sum",
             None),
            ("L1 pending stall cycles", "TCP_PENDING_STALL_CYCLES_sum", None),
            ("GPU busy cycles (GRBM_GUI_ACTIVE)", "GRBM_GUI_ACTIVE", None)]
    orders = [o for o in ("entry", "layer") if any(key[0] == o for key in per)]
    head = "| per launch | " + " | ".join(f"gather ({o})" for o in orders) + " | " + \
        " | ".join(f"scatter ({o})" for o in orders) + " |"
    lines += [head, "|---|" + "---|" * (2 * len(orders))]
    for label, c, denom in rows:
        cells = []
        for k in ("gather", "scatter"):
            for o in orders:
                x = v(o, k, c) / v(o, k, denom) if denom else v(o, k, c)
                cells.append(f"{x:,.1f}" if denom else f"{x:,.0f}")
        lines.append(f"| {label} | " + " | ".join(cells) + " |")
    open(HBM_COUNTERS_SUMMARY, "w").write("\n".join(lines) + "\n")
    print(open(HBM_COUNTERS_SUMMARY).read())


HASH_SUMMARY = os.path.join(ROOT, "profiles", "sha256_hash_workloads_kernel_trace.md")
HASH_BYTES_SUMMARY = os.path.join(ROOT, "profiles", "sha256_hash_batch_hbm_bytes.md")
HASH_SOURCE = os.path.join(ROOT, "paper_2609_33762_amd", "csrc", "ea_sha256_kernels.hip")
# the hash line's roofline case: 65,536 sequences of 256 tokens, 16-token blocks
HASH_BATCH = (65536, 256, 16)


def hash_source_hash():
    return hashlib.sha256(open(HASH_SOURCE, "rb").read()).hexdigest()[:16]


def hash_batch_bytes():
    """Algorithmic bytes of one call of the batch case with offsets in HBM:
    the tokens and the sequence offsets read once, the key offsets and the
    keys written once."""
    n, t, b = HASH_BATCH
    return n * t * 4 + (n + 1) * 8 + (n + 1) * 8 + n * (t // b) * 32


def hash_traffic():
    """HBM bytes per call of the batch case from the committed counter
    summary, or None when it is missing or was taken from other hash kernel
    sources."""
    if not os.path.exists(HASH_BYTES_SUMMARY):
        return None
    src = val = None
    for line in open(HASH_BYTES_SUMMARY):
        if line.startswith("hash_kernel_source_sha256:"):
            src = line.split(":", 1)[1].strip()
        if line.startswith("traffic_bytes_per_call:"):
            val = int(line.split(":", 1)[1])
    return val if src == hash_source_hash() else None
HASH_CASE_NOTES = {
    "turn_56k_prompt": "the turn's 56,000-token prompt as one chain",
    "turn_56k_prompt_1024_token_chunks": "the same prompt in 1,024-token chunks (64 token "
                                         "blocks per key)",
    "one_64k": "one 65,536-token sequence",
    "pool_64x64k": "64 sequences of 65,536 tokens",
    "batch_16384x1k": "16,384 sequences of 1,024 tokens",
    "batch_65536x256": "65,536 sequences of 256 tokens",
}


def _hash_role(name):
    n = _plain_name(name)
    return n if ("sha256" in n or "hash_" in n) else None


def _hash_counter_calls(path, ctr):
    """Per-call counter values of the hash kernels in a counter-collection
    CSV, in dispatch order: each call ends with its chain or fused kernel."""
    rows = [x for x in csv.DictReader(open(path)) if x["Counter_Name"] == ctr]
    rows.sort(key=lambda x: int(x["Dispatch_Id"]))
    calls, cur = [], []
    for x in rows:
        role = _hash_role(x["Kernel_Name"])
        if role is None:
            continue
        cur.append((role, float(x["Counter_Value"])))
        if "chain" in role or "fused" in role:
            calls.append(cur)
            cur = []
    return calls


def _hash_series(line, calls, case_name, kind):
    """The timed calls of one series, located with the counts the line
    records (each case: the host entry point's check call, then each
    series' untimed and timed calls)."""
    want = sum(1 + sum(sum(c) for c in case["calls"].values()) for case in line["hash"].values())
    if len(calls) != want:
        raise SystemExit(f"{len(calls)} calls in the counters, the run made {want}")
    i = 0
    for name, case in line["hash"].items():
        i += 1
        for k, (n_untimed, n_timed) in case["calls"].items():
            if name == case_name and k == kind:
                return calls[i + n_untimed:i + n_untimed + n_timed]
            i += n_untimed + n_timed
    raise SystemExit(f"no series {case_name}/{kind} in the line")


def summarize_hash_bytes(d):
    """Write the HBM byte summary of the hash line's roofline case from two
    rocprofv3 counter runs of `bench.py --workload hash` under d (FETCH_SIZE
    in d/prof_hash_fetch, WRITE_SIZE in d/prof_hash_write, each beside the
    line its run printed), scaled like the piece-copy counters."""
    import re
    m = re.search(r"FETCH_SIZE is scaled by ([0-9.]+) and WRITE_SIZE by ([0-9]+\.[0-9]+)",
                  open(TRAFFIC_SUMMARY).read())
    cal = {"FETCH_SIZE": float(m.group(1)), "WRITE_SIZE": float(m.group(2))}
    per = {}
    for label, ctr in (("fetch", "FETCH_SIZE"), ("write", "WRITE_SIZE")):
        base = os.path.join(d, f"prof_hash_{label}")
        line = json.load(open(os.path.join(base, "hash.json")))
        calls = _hash_counter_calls(os.path.join(base, f"{label}_counter_collection.csv"), ctr)
        series = _hash_series(line, calls, "batch_65536x256", "device_offsets")
        kernels = {}
        for call in series:
            for role, v in call:
                kernels.setdefault(role, []).append(v)
        per[ctr] = {k: float(np.median(v)) for k, v in kernels.items()}
    roles = sorted(set(per["FETCH_SIZE"]) | set(per["WRITE_SIZE"]))
    total = sum((per["FETCH_SIZE"].get(k, 0.0) * cal["FETCH_SIZE"] +
                 per["WRITE_SIZE"].get(k, 0.0) * cal["WRITE_SIZE"]) * 1024 for k in roles)
    alg = hash_batch_bytes()
    n, t, b = HASH_BATCH
    cmd = ("rocprofv3 --pmc {c} --output-format csv -d bench_out/prof_hash_{l} -o {l} -- "
           "python3 -u bench.py --workload hash > bench_out/prof_hash_{l}/hash.json")
    lines = [f"# HBM bytes per call: chained keys of {n:,} sequences of {t} tokens "
             f"({b}-token blocks, offsets in HBM)", "",
             "Commands (from the repository root on the MI355X):", "",
             "    " + cmd.format(c="FETCH_SIZE", l="fetch"),
             "    " + cmd.format(c="WRITE_SIZE", l="write"),
             "    python3 bench.py --summarize-hash-bytes bench_out", "",
             f"hash_kernel_source_sha256: {hash_source_hash()}", "",
             "The 20 timed calls of the batch case with device offsets (the hash line's "
             "roofline case), median per kernel over the calls.  Counters are scaled as in "
             f"the piece-copy summary (FETCH_SIZE x{cal['FETCH_SIZE']:.3f}, WRITE_SIZE "
             f"x{cal['WRITE_SIZE']:.3f}).", "",
             "| kernel | FETCH_SIZE KiB | WRITE_SIZE KiB | scaled bytes |", "|---|---|---|---|"]
    for k in roles:
        f, w = per["FETCH_SIZE"].get(k, 0.0), per["WRITE_SIZE"].get(k, 0.0)
        lines.append(f"| {k} | {f:.0f} | {w:.0f} | "
                     f"{(f * cal['FETCH_SIZE'] + w * cal['WRITE_SIZE']) * 1024:.0f} |")
    lines += ["", f"Per call: {total:.0f} bytes against {alg} algorithmic (tokens and sequence "
              f"offsets read once, key offsets and keys written once): ratio "
              f"{total / alg:.4f}.", "", f"traffic_bytes_per_call: {total:.0f}"]
    open(HASH_BYTES_SUMMARY, "w").write("\n".join(lines) + "\n")
    print(open(HASH_BYTES_SUMMARY).read())


def summarize_hash(d):
    """Write the hash kernel summary from directory d: the line printed by
    `bench.py --workload hash` (hash.json) and the kernel trace of the same
    run (hash_kernel_trace.csv).  The trace is cut into calls (each call
    ends with its chain or fused kernel), and the calls into the run's
    series with the counts the line records."""
    line = json.load(open(os.path.join(d, "hash.json")))
    rows = sorted(csv.DictReader(open(os.path.join(d, "hash_kernel_trace.csv"))),
                  key=lambda x: int(x["Start_Timestamp"]))
    calls, cur = [], []
    for x in rows:
        role = _hash_role(x["Kernel_Name"])
        if role is None:
            continue
        wg = int(x["Grid_Size_X"]) // max(1, int(x["Workgroup_Size_X"]))
        dur = (int(x["End_Timestamp"]) - int(x["Start_Timestamp"])) / 1e3
        cur.append((role, wg, int(x["Workgroup_Size_X"]), dur))
        if "chain" in role or "fused" in role:
            calls.append(cur)
            cur = []
    want = sum(1 + sum(sum(c) for c in case["calls"].values()) for case in line["hash"].values())
    if len(calls) != want:
        raise SystemExit(f"{len(calls)} calls in the trace, the run made {want}")
    lines = ["# Hash kernels on the hash workload (kernel trace)", "",
             "Command (from the repository root on the MI355X):", "",
             "    rocprofv3 --kernel-trace --stats --output-format csv -d bench_out/prof_hash "
             "-o hash -- python3 -u bench.py --workload hash > bench_out/prof_hash/hash.json",
             "    python3 bench.py --summarize-hash bench_out/prof_hash", "",
             "`bench.py --workload hash` runs six cases of chained keys (16-token blocks unless "
             "named otherwise, tokens already in HBM).  Per case it first checks the keys of one "
             "call of the host entry point, then times two series of 20 back-to-back calls "
             "between one pair of HIP events, each after 0.3 s of untimed calls: "
             "`ea_hash_blocks_device_offsets` (sequence offsets in HBM, key offsets from the "
             "library's scan kernels) and `ea_hash_blocks_device` (host offsets uploaded by each "
             "call).  The tables give the median duration of each kernel over the 20 timed "
             "calls, their sum, and the HIP-event time per call the bench reports.  Grids are "
             "in workgroups (work-items per workgroup in parentheses).", ""]
    i = 0
    summary = []
    for name, case in line["hash"].items():
        i += 1  # the host entry point's checking call
        series = {}
        for kind in ("device_offsets", "host_offsets"):
            n_untimed, n_timed = case["calls"][kind]
            i += n_untimed
            series[kind] = calls[i:i + n_timed]
            i += n_timed
        lines += [f"## {name}: {HASH_CASE_NOTES.get(name, name)} ({case['keys']:,} keys)", "",
                  "| series | kernel (grid) | median µs |", "|---|---|---|"]
        for kind, ev in (("device_offsets", case["ms"]), ("host_offsets", case["ms_host_offsets"])):
            per = {}
            for c in series[kind]:
                for role, wg, wgs, dur in c:
                    per.setdefault((role, wg, wgs), []).append(dur)
            tot = float(np.median([sum(x[3] for x in c) for c in series[kind]]))
            for (role, wg, wgs), v in per.items():
                lines.append(f"| {kind} | {role} ({wg:,} x {wgs}) | {np.median(v):.1f} |")
            lines.append(f"| {kind} | kernels of one call | {tot:.1f} |")
            lines.append(f"| {kind} | one call, HIP events | {ev * 1e3:.1f} |")
            summary.append((name, kind, tot, ev * 1e3, case["keys"]))
        lines.append("")
    lines += ["## Per key", "", "| case | series | kernels µs per key | call µs per key |",
              "|---|---|---|---|"]
    for name, kind, tot, ev, keys in summary:
        lines.append(f"| {name} | {kind} | {tot / keys:.4f} | {ev / keys:.4f} |")
    roof = line["roofline"]
    lines += ["", f"Roofline case (the line's `roofline`): {roof['kernel']}: {roof['achieved']} "
              f"{roof['unit']} against {roof['peak']} ({roof['frac']:.1%}).", ""]
    open(HASH_SUMMARY, "w").write("\n".join(lines))
    print("\n".join(lines))


def _quiet_cache(torch, api, sh, num_pages=None):
    """A cache of shape sh (contents irrelevant for timing: left unfilled)."""
    P = num_pages or sh.num_pages
    kv = torch.empty(sh.num_layers * P * sh.piece_bytes, dtype=torch.uint8, device="cuda")
    cache = api.Cache(kv, P, sh.num_layers, sh.page_tokens, sh.num_kv_heads, sh.head_dim,
                      sh.elem_bytes)
    return kv, cache


def run_load_cost(args):
    """Restore cost of Eq. 2, T_load(n) = n beta / B_eff + tau_load, fitted
    from load sweeps on the Qwen3 turn shape (96 KiB/token), the dense shape
    (128 KiB/token), one TP8 rank of Qwen3 (24 KiB/token) with 16-token slots
    and with 1,024-token chunks.  Each point is the median of repeated loads
    of n random resident slots into random free pages, timed on the device
    (HIP events) and end to end (call to completion on the host clock)."""
    import torch
    from paper_2609_33762_amd import api, drivers, workloads as W
    torch.cuda.set_device(0)
    cur = torch.cuda.current_stream()
    setups = [
        ("qwen3_96KiB_per_token", W.QWEN3, 1, [1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024, 1500]),
        ("dense_128KiB_per_token", W.DENSE, 1, [1, 2, 3, 4, 5, 6, 7, 8, 16, 64, 256, 1024]),
        ("qwen3_tp8_24KiB_per_token", W.QWEN3_TP8, 1,
         [1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024, 1500]),
        ("qwen3_tp8_1024_token_chunks", W.QWEN3_TP8, W.CHUNK_PAGES, [1, 2, 4, 8, 16, 23]),
    ]
    r = W.rng(W.SEED_IDS)
    res = {}
    for name, sh, C, sizes in setups:
        kv, cache = _quiet_cache(torch, api, sh)
        beta = sh.num_layers * sh.piece_bytes // sh.page_tokens
        top = max(sizes)
        tier = api.Tier(cache, top * C * sh.num_layers * sh.piece_bytes + 4096, chunk_pages=C)
        assert tier.capacity >= top
        src = W.distinct(r, sh.num_pages, top * C)
        tier.store(cache, src, np.arange(top), stream=cur)
        torch.cuda.synchronize()
        pts = drivers.load_cost_sweep(torch, cache, tier, sh, sizes, cur, r)
        tier.close()
        cache.close()
        del kv
        torch.cuda.empty_cache()
        tok = np.array([p[0] for p in pts], np.float64)
        nb = tok * beta
        fits = {}
        for k, col in (("device", 2), ("end_to_end", 3)):
            B, tau, resid = drivers.fit_load_cost(nb, np.array([p[col] for p in pts]) * 1e-3)
            fits[k] = {"B_eff_gbs": round(float(B) / GB, 2), "tau_load_us": round(float(tau) * 1e6, 1),
                       "us_per_token_large_n": round(float(beta / B) * 1e6, 4),
                       "max_rel_residual": round(resid, 3)}
        res[name] = {"beta_bytes_per_token": beta, "chunk_pages": C, "fit": fits,
                     "points_tokens_bytes_devms_wallms": [[int(a), int(b), round(c, 4), round(d, 4)]
                                                         for a, b, c, d in pts]}
        log(f"{name}: {fits}")
    head = res["qwen3_96KiB_per_token"]["fit"]["device"]
    return _line("load_cost: load sweeps, T_load(n) = n beta / B_eff + tau_load fitted at "
                 "96/128/24 KiB per token and 1,024-token chunks", head["B_eff_gbs"], "GB/s",
                 None, sum(len(x[3]) for x in setups), {"load_cost": res})


RESTORE_FIT_SIZES = [1, 4, 16, 64, 256, 1024, 1500]
RESTORE_FIT_REPS = 5
RESTORE_FIT_LOADS = len(RESTORE_FIT_SIZES) * RESTORE_FIT_REPS


def restore_fit(peak_h2d):
    """Eq. 2's restore cost on one TP8 rank's shard of the Qwen3 KV (1 KV
    head, 24 KiB per token), the per-rank setting of the paper's H20 figure:
    a short sweep of loads (1 to 1,500 random resident slots into random
    free pages, medians of 5) fitted to T_load(n) = n beta / B_eff + tau."""
    import torch
    from paper_2609_33762_amd import api, drivers, workloads as W
    sh = W.QWEN3_TP8
    cur = torch.cuda.current_stream()
    kv, cache = _quiet_cache(torch, api, sh)
    beta = sh.num_layers * sh.piece_bytes // sh.page_tokens
    sizes = RESTORE_FIT_SIZES
    top = max(sizes)
    tier = api.Tier(cache, top * sh.num_layers * sh.piece_bytes + 4096)
    r = W.rng(W.SEED_IDS)
    tier.store(cache, W.distinct(r, sh.num_pages, top), np.arange(top), stream=cur)
    torch.cuda.synchronize()
    rows = drivers.load_cost_sweep(torch, cache, tier, sh, sizes, cur, r, reps=RESTORE_FIT_REPS)
    tier.close()
    cache.close()
    del kv
    torch.cuda.empty_cache()
    tok = np.array([x[0] for x in rows], np.float64)
    out = {"shape": "Qwen3-30B-A3B KV on one TP8 rank: 1 KV head, 24 KiB per token, "
                    "16-token slots of 384 KiB",
           "sweep_pages": sizes}
    for k, col in (("device", 2), ("end_to_end", 3)):
        B, tau, resid = drivers.fit_load_cost(tok * beta, np.array([x[col] for x in rows]) * 1e-3)
        out[k] = {"B_eff_gbs": round(B / GB, 2), "tau_load_us": round(tau * 1e6, 1),
                  "us_per_token_per_rank": round(beta / B * 1e6, 4),
                  "frac_of_h2d_peak": round(B / GB / peak_h2d, 4),
                  "max_rel_residual": round(resid, 3)}
    out["context_h20_us_per_token_per_rank"] = 0.86
    return out


PLAN_CASES = (
    # name, shape, chunk pages, pages per call (store / load), calls timed
    ("qwen3_turn", "QWEN3", 1, 2000, 1500, 3),
    ("tp8_shard", "QWEN3_TP8", 1, 2000, 1500, 3),
    ("tp8_chunks_1024_tokens", "QWEN3_TP8", 64, 31, 23, 3),
    ("layered_fp8_prefix", "LAYERED", 1, 4096, 4096, 3),
    ("dense_8_pages", "DENSE", 1, 8, 8, 50),
    ("dense_4_pages", "DENSE", 1, 4, 4, 50),
    ("dense_1_page", "DENSE", 1, 1, 1, 50),
)


def run_plans(args):
    """Stores and loads alone under one transfer plan (--plan direct or
    staged) for each size class the workloads use: the Qwen3 turn (2,000 /
    1,500 pages of 1.5 MiB), one TP8 rank's turn (384 KiB pages, and the
    paper's 1,024-token chunks of 24 MiB), the layered fp8 prefix (768 KiB
    pages with scales) and the dense model's calls of 8, 4 and 1 pages of
    2 MiB; each first to consecutive slots, then to random ones.  Direct:
    one kernel between the cache and the mapped pinned slots.  Staged: a
    paged gather or scatter through an HBM staging buffer plus
    hipMemcpyAsync of each run of consecutive slots.  Each operation is two
    untimed calls (the second right before the start event) and then the
    timed ones between HIP events.  Caches are
    left unfilled (contents do not change the timing), so the only copy
    kernels in the process are the plan's own: a rocprofv3 run of this
    command attributes its kernels and byte counters to the plan."""
    import torch
    from paper_2609_33762_amd import api, _native as N, workloads as W
    torch.cuda.set_device(0)
    plan_name = "staged" if args.plan == "staged" else "direct"
    plan = N.EA_PLAN_STAGED if plan_name == "staged" else N.EA_PLAN_DIRECT
    cur = torch.cuda.current_stream()
    out, link = {}, 0
    for name, shape, C, n_s, n_l, reps in PLAN_CASES:
        sh = getattr(W, shape)
        r = W.rng(W.SEED_IDS)
        P = sh.num_pages
        kv = torch.empty(sh.cache_bytes, dtype=torch.uint8, device="cuda")
        sc = torch.empty(sh.num_layers * P * 8, dtype=torch.uint8, device="cuda") \
            if sh.has_scales else None
        cache = api.Cache(kv, P, sh.num_layers, sh.page_tokens, sh.num_kv_heads, sh.head_dim,
                          sh.elem_bytes, scales=sc)
        slot_pages = sh.num_layers * sh.piece_bytes * C + (4096 if sh.has_scales else 0)
        cap_slots = max(2 * n_s, 64)
        tier = api.Tier(cache, cap_slots * slot_pages, chunk_pages=C)
        tier.set_plan(N.EA_DIR_BOTH, plan)
        src = W.distinct(r, P, n_s * C)
        dst = W.distinct(r, P, n_l * C, exclude=src)
        page = tier.slot_bytes
        res = {}
        for slots_name, slots in (("consecutive", np.arange(n_s, dtype=np.int64)),
                                  ("random", W.distinct(r, tier.capacity, n_s))):
            st = event_ms(torch, lambda: tier.store(cache, src, slots, stream=cur), cur, reps)
            ld = event_ms(torch, lambda: tier.load(cache, slots[:n_l], dst, stream=cur), cur,
                          reps)
            res[slots_name] = {"store_ms": round(st, 4),
                               "store_gbs": round(n_s * page / st / 1e6, 2),
                               "load_ms": round(ld, 4), "load_gbs": round(n_l * page / ld / 1e6, 2)}
            link += (2 + reps) * (n_s + n_l) * page
        out[name] = {"slot_bytes": page, "store_slots": n_s, "load_slots": n_l, **res}
        log(f"plan {plan_name}, {name}: {res}")
        torch.cuda.synchronize()
        tier.close()
        cache.close()
        del kv, sc
        torch.cuda.empty_cache()
    return _line(f"plans: stores and loads alone per size class, {plan_name} plan, consecutive and "
                 "random slots", out["qwen3_turn"]["random"]["store_gbs"], "GB/s", None, 3,
                 {"plan": plan_name, "plans": out, "link_bytes_all_calls": link})


def summarize_plans(d):
    """The plan summary in profiles/ from three rocprofv3 runs (kernel
    trace, FETCH_SIZE, WRITE_SIZE) of each plan's `--workload plans` command,
    under d/plans_<plan>/, beside the runs' own JSON lines."""
    import re
    m = re.search(r"FETCH_SIZE is scaled by ([0-9.]+) and WRITE_SIZE by ([0-9]+\.[0-9]+)",
                  open(TRAFFIC_SUMMARY).read())
    cal_f, cal_w = float(m.group(1)), float(m.group(2))
    lines = ["# Transfer plans: direct kernels against HBM staging plus hipMemcpyAsync, per "
             "size class", "",
             "Commands (from the repository root on the MI355X), for P in direct and staged:", "",
             "    rocprofv3 --kernel-trace --memory-copy-trace --stats --output-format csv "
             "-d bench_out/plans_P/trace -o trace -- python3 bench.py --workload plans --plan P",
             "    rocprofv3 --pmc FETCH_SIZE --output-format csv -d bench_out/plans_P/fetch -o fetch "
             "-- python3 bench.py --workload plans --plan P",
             "    rocprofv3 --pmc WRITE_SIZE --output-format csv -d bench_out/plans_P/write -o write "
             "-- python3 bench.py --workload plans --plan P",
             "    python3 bench.py --workload plans --plan P > bench_out/plans_P/line.json",
             "    python3 bench.py --summarize-plans bench_out", "",
             f"kernel_source_sha256: {kernel_source_hash()}", "",
             "Each process runs one plan over every size class: stores and loads alone, to "
             "consecutive slots and then to random ones, two untimed calls and then the timed "
             "ones.  Every copy kernel in a process belongs to its plan, apart from the few "
             "bytes the library's one-time XCD probe copies back.  Byte counters are "
             f"scaled as in the piece-copy summary (FETCH_SIZE x{cal_f:.3f}, WRITE_SIZE "
             f"x{cal_w:.3f}) and include the host-memory side.", ""]
    both = {plan: json.load(open(os.path.join(d, f"plans_{plan}", "line.json")))["plans"]
            for plan in ("direct", "staged")}
    lines += ["## Rates per size class (HIP events, GB/s; store / load)", "",
              "From the run without the profiler (the last command before the summary): the "
              "copy trace adds its own cost to each of the staged plan's many small copies.", "",
              "| case | slot bytes | slots per call (store / load) | direct, consecutive | "
              "staged, consecutive | direct, random | staged, random |", "|---|---|---|---|---|---|---|"]
    for case, v in both["direct"].items():
        w = both["staged"][case]
        cell = lambda x, k: f"{x[k]['store_gbs']} / {x[k]['load_gbs']}"  # noqa: E731
        lines.append(f"| {case} | {v['slot_bytes']} | {v['store_slots']} / {v['load_slots']} | "
                     f"{cell(v, 'consecutive')} | {cell(w, 'consecutive')} | "
                     f"{cell(v, 'random')} | {cell(w, 'random')} |")
    lines.append("")
    for plan in ("direct", "staged"):
        base = os.path.join(d, f"plans_{plan}")
        res = json.load(open(os.path.join(base, "line.json")))
        lines += [f"## {plan}", ""]
        lines += ["", "| kernel | calls | total ms | avg ms |", "|---|---|---|---|"]
        for x in csv.DictReader(open(os.path.join(base, "trace", "trace_kernel_stats.csv"))):
            name = x["Name"]
            if "copy_host_link" in name or "copy_hbm" in name or "__amd_rocclr" in name:
                short = name.replace("void ", "").replace("ea::(anonymous namespace)::", "")
                short = short.split("(")[0]
                lines.append(f"| `{short}` | {x['Calls']} | {int(x['TotalDurationNs']) / 1e6:.2f} | "
                             f"{float(x['AverageNs']) / 1e6:.4f} |")
        mc = os.path.join(base, "trace", "trace_memory_copy_trace.csv")
        copies = list(csv.DictReader(open(mc))) if os.path.exists(mc) else []
        lost = None
        log_f = os.path.join(base, "trace.log")
        if os.path.exists(log_f):
            m2 = re.search(r"(\d+) completion callbacks were not delivered", open(log_f).read())
            lost = int(m2.group(1)) if m2 else None
        if copies:
            dur = sum(int(x["End_Timestamp"]) - int(x["Start_Timestamp"]) for x in copies) / 1e6
            dirs = sorted({x["Direction"] for x in copies})
            lines += ["", f"Copies the runtime ran on its copy engines (not kernels, so absent "
                      f"from the kernel table and the byte counters): {len(copies)} copies "
                      f"({', '.join(dirs)}), {dur:.2f} ms in total."]
            if lost:
                lines += [f"The copy trace is incomplete: rocprofv3 reported {lost} completion "
                          "callbacks of the copies never delivered, so these counts and times "
                          "are lower bounds."]
        elif plan == "staged":
            lines += ["", "No copy ran on the copy engines: every hipMemcpyAsync was a blit "
                      "kernel."]
        counters = {label: os.path.join(base, label, f"{label}_counter_collection.csv")
                    for label in ("fetch", "write")}
        if not all(os.path.exists(f) for f in counters.values()):
            lines += ["", "Byte counters: not collected for this plan in this retake (its "
                      "FETCH_SIZE pass stopped with a segmentation fault in host code, inside "
                      "the profiler's interception of the plan's own runtime calls).", ""]
            continue
        tot = {}
        for label, ctr in (("fetch", "FETCH_SIZE"), ("write", "WRITE_SIZE")):
            s = 0.0
            for x in csv.DictReader(open(counters[label])):
                n = x["Kernel_Name"]
                if x["Counter_Name"] == ctr and ("copy_host_link" in n or "copy_hbm" in n or
                                                  "__amd_rocclr" in n):
                    s += float(x["Counter_Value"])
            tot[ctr] = s
        traffic = (tot["FETCH_SIZE"] * cal_f + tot["WRITE_SIZE"] * cal_w) * 1024
        link = res["link_bytes_all_calls"]
        lines += ["", f"Memory traffic of the plan's kernels over all calls: {traffic / 1e9:.2f} GB "
                  f"for {link / 1e9:.2f} GB across the host link, {traffic / link:.2f} bytes per "
                  "link byte (each byte read once and written once is 2.00"
                  + (", and copies on the copy engines add traffic the counters do not see"
                     if copies else "") + ").", ""]
    open(PLANS_SUMMARY, "w").write("\n".join(lines) + "\n")
    print(open(PLANS_SUMMARY).read())


def run_tp8_shard(args):
    """One Qwen3 turn on a TP8 rank's share (1 KV head, 24 KiB/token):
    a 2,000-page refill stored and a 1,500-page prefix loaded, alone and
    together on two streams, with 16-token slots and with 1,024-token chunks
    (31 and 23 chunks of 24 MiB)."""
    import torch
    from paper_2609_33762_amd import api, workloads as W
    torch.cuda.set_device(0)
    sh = W.QWEN3_TP8
    r = W.rng(W.SEED_IDS)
    kv, cache = _quiet_cache(torch, api, sh)
    W.fill_bf16_normal(kv, W.SEED_DATA)
    beta = sh.num_layers * sh.piece_bytes // sh.page_tokens
    out = {}
    for C, n_s, n_l in ((1, 2000, 1500), (W.CHUNK_PAGES, 31, 23)):
        tier = api.Tier(cache, W.QWEN3_TIER_BYTES, chunk_pages=C)
        prefix = W.distinct(r, sh.num_pages, n_l * C)
        refill = W.distinct(r, sh.num_pages, n_s * C, exclude=prefix)
        dst = W.distinct(r, sh.num_pages, n_l * C, exclude=np.concatenate([prefix, refill]))
        pslots = np.arange(n_l)
        sslots = np.arange(n_l, n_l + n_s)
        tier.store(cache, prefix, pslots)
        torch.cuda.synchronize()
        cur = torch.cuda.current_stream()
        st_ms = event_ms(torch, lambda: tier.store(cache, refill, sslots, stream=cur), cur, 5)
        ld_ms = event_ms(torch, lambda: tier.load(cache, pslots, dst, stream=cur), cur, 5)
        s_store, s_load = copy_streams(torch)
        both = []
        for _ in range(5):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            tier.load(cache, pslots, dst, stream=s_load)
            tier.store(cache, refill, sslots, stream=s_store)
            torch.cuda.synchronize()
            both.append(time.perf_counter() - t0)
        sb, lb = n_s * tier.slot_bytes, n_l * tier.slot_bytes
        key = "page_slots" if C == 1 else "chunk_slots_1024_tokens"
        out[key] = {"slot_bytes": tier.slot_bytes, "store_slots": n_s, "load_slots": n_l,
                    "store_gbs": round(sb / (st_ms * 1e-3) / GB, 2),
                    "load_gbs": round(lb / (ld_ms * 1e-3) / GB, 2),
                    "duplex_gbs": round((sb + lb) / float(np.median(both)) / GB, 2),
                    "load_us_per_token": round(ld_ms * 1e3 / (n_l * C * sh.page_tokens), 4)}
        log(f"tp8 shard, {key}: {out[key]}")
        tier.close()
    cache.close()
    del kv
    torch.cuda.empty_cache()
    return _line("tp8_shard: Qwen3 turn on one TP8 rank (24 KiB/token), 16-token slots and "
                 "1,024-token chunks", out["page_slots"]["duplex_gbs"], "GB/s", None, 5,
                 {"tp8_shard": out, "beta_bytes_per_token": beta})


# Lane-instructions per key with 16-token blocks in one-lane form, counted
# in the library's gfx950 assembly (loop bodies): 1,410 for the token block
# (sha256_midstates) and 1,378 for the chained compression
# (sha256_chain_lane).  This is the work of a key; the two-lane chain form
# issues 2 x 1,162 lane-instructions for the same compression, and that
# surplus counts as overhead, not as work.
HASH_INSTR_PER_KEY = 1410 + 1378
# Integer VALU peak of MI355X: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz (a
# wave64 instruction occupies a SIMD for 4 cycles; the 157.3 TFLOP/s fp32
# figure counts packed two-wide FMAs, which integer ops do not have).
VALU_INT_PEAK = 256 * 4 * 16 * 2.4e9


def run_hash(args):
    """Chained keys (16-token blocks) on the device, tokens already in HBM:
    the turn's 56k-token prompt (one 3,500-key chain, and in 1,024-token
    chunks: 54 keys of 64 token blocks each), one 64k-token sequence, 64
    such sequences (these three in the two-wave form, one workgroup per
    sequence), 16,384 sequences of 1,024 tokens (the two-lane chain kernel
    then has 512 waves for the 1,024 SIMDs) and 65,536 of 256 tokens (more
    than 32 sequences per SIMD, so the chain runs one lane per sequence:
    1,024 waves); every run checked against the host entry point's keys.
    The roofline is taken on the last."""
    import torch
    torch.cuda.set_device(0)
    out = {}
    for name, lengths, b in (("turn_56k_prompt", [56000], 16),
                             ("turn_56k_prompt_1024_token_chunks", [56000], 1024),
                             ("one_64k", [65536], 16), ("pool_64x64k", [65536] * 64, 16),
                             ("batch_16384x1k", [1024] * 16384, 16),
                             ("batch_65536x256", [256] * 65536, 16)):
        out[name] = hash_case(torch, lengths, b)
        log(f"hash {name}: {out[name]}")
    b = out["batch_65536x256"]
    roof = hash_roofline(b)
    extra = {"hash": out, "roofline": roof}
    if not args.no_cpu_baseline:
        from paper_2609_33762_amd import workloads as W
        extra["cpu_baseline"] = _hash_cpu_baseline(W)
        log(f"cpu baseline: {extra['cpu_baseline']}")
    return _line("hash: chained SHA-256 keys of 16-token blocks, tokens in HBM",
                 round(b["tokens_per_s"] / 1e9, 3), "G tokens/s", b["ms"], 20, extra)


def hash_roofline(b):
    """The hash roofline on the 65,536 x 256-token case b (device offsets)."""
    achieved = b["keys"] * HASH_INSTR_PER_KEY / (b["ms"] * 1e-3)
    return {"bound": "alu", "kernel": "hash_offsets_partials + sha256_fused_scan "
                                      "(65,536 x 256 tokens, offsets in HBM)",
            "achieved": round(achieved / 1e12, 3), "peak": round(VALU_INT_PEAK / 1e12, 2),
            "unit": "T lane-instructions/s", "frac": round(achieved / VALU_INT_PEAK, 4),
            "traffic": hash_traffic(), "traffic_algorithmic": hash_batch_bytes()}


def hash_case(torch, lengths, b):
    """One hash case: sequences of the given lengths, keys of b-token blocks,
    tokens already in HBM, checked against the host entry point's keys, then
    timed with device offsets and with host offsets (20 calls each between
    one pair of HIP events after 0.3 s of untimed calls)."""
    from paper_2609_33762_amd import api, workloads as W
    cur = torch.cuda.current_stream()
    toks, offs = W.sequences(W.SEED_TOKENS, lengths)
    d_tok = torch.as_tensor(toks, device="cuda")
    d_offs = torch.as_tensor(offs, device="cuda")
    d_koffs = torch.empty(len(offs), dtype=torch.int64, device="cuda")
    nk = int(sum(n // b for n in lengths))
    d_keys = torch.empty(nk * 32, dtype=torch.uint8, device="cuda")
    host, _ = api.hash_blocks(toks, offs, b)
    # tokens and offsets resident in HBM (the key offsets from the scan
    # kernel), and for comparison host offsets uploaded by each call
    calls = {"device_offsets": lambda: api.hash_blocks_device_offsets(  # noqa: E731
                 d_tok, d_offs, b, d_keys, d_koffs, stream=cur),
             "host_offsets": lambda: api.hash_blocks_device(  # noqa: E731
                 d_tok, offs, b, d_keys, stream=cur)}
    res, counts = {}, {}
    for kind, call in calls.items():
        # untimed calls for 0.3 s first: a GPU left idle or lightly loaded
        # runs at lower clocks and takes a while to rise (successive single
        # chains measured 2.8 down to 2.1 us per key)
        t_warm = time.perf_counter() + 0.3
        n_warm = 0
        while time.perf_counter() < t_warm:
            call()
            torch.cuda.synchronize()
            n_warm += 1
        d_keys.zero_()
        ms = event_ms(torch, call, cur, 20, warm=2)
        assert np.array_equal(host, d_keys.cpu().numpy().reshape(-1, 32)), (lengths[:2], kind)
        res[kind] = ms
        # calls in launch order (untimed, timed): a kernel trace of the
        # run is cut into calls with these counts
        counts[kind] = [n_warm + 3, 20]
    ms = res["device_offsets"]
    return {"ms": round(ms, 4), "ms_host_offsets": round(res["host_offsets"], 4),
            "keys": nk, "us_per_key": round(ms * 1e3 / nk, 4),
            "tokens_per_s": round(sum(lengths) / (ms * 1e-3), 1), "calls": counts}


def _hash_cpu_baseline(W):
    """The oracle on one core: the turn's 56,000-token prompt as one chain,
    and 1,024 of the batch's 256-token sequences (medians of 5)."""
    import oracle

    def run():
        res = {}
        for name, lengths in (("turn_56k_prompt", [56000]), ("batch_1024x256", [256] * 1024)):
            toks, offs = W.sequences(W.SEED_TOKENS, lengths)
            ts = []
            for _ in range(5):
                t0 = time.perf_counter()
                oracle.hash_blocks(toks, offs, 16)
                ts.append(time.perf_counter() - t0)
            res[name] = sum(lengths) / float(np.median(ts))
        return res

    res = _pinned_one_core(run)
    return {"value": round(res["batch_1024x256"] / 1e9, 5), "unit": "G tokens/s", "cores": 1,
            "kind": "oracle", "turn_56k_prompt_ms": round(56000 / res["turn_56k_prompt"] * 1e3, 3),
            "sample": "the turn's 56,000-token prompt as one chain, and 1,024 sequences of 256 "
                      "tokens (a 64th of the batch), medians of 5"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--plan", choices=["auto", "direct", "staged"], default="auto")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--isolated-only", action="store_true")
    ap.add_argument("--summarize-profiles", metavar="DIR")
    ap.add_argument("--summarize-plans", metavar="DIR")
    ap.add_argument("--summarize-workloads", metavar="DIR")
    ap.add_argument("--summarize-hbm-counters", metavar="DIR")
    ap.add_argument("--summarize-hash", metavar="DIR")
    ap.add_argument("--summarize-hash-bytes", metavar="DIR")
    ap.add_argument("--workload", default="qwen3_turn",
                    choices=["qwen3_turn", "agent_pool", "dense_scattered", "layered_fp8", "tiny",
                             "load_cost", "tp8_shard", "hash", "agent_pool_chunked", "plans"])
    ap.add_argument("--turns-per-agent", type=int, default=24)
    ap.add_argument("--detail", default=os.path.join(ROOT, "bench_out", "bench_detail.json"))
    args = ap.parse_args()
    if args.summarize_profiles:
        summarize_profiles(args.summarize_profiles)
        return
    if args.summarize_plans:
        summarize_plans(args.summarize_plans)
        return
    if args.summarize_workloads:
        summarize_workloads(args.summarize_workloads)
        return
    if args.summarize_hbm_counters:
        summarize_hbm_counters(args.summarize_hbm_counters)
        return
    if args.summarize_hash:
        summarize_hash(args.summarize_hash)
        return
    if args.summarize_hash_bytes:
        summarize_hash_bytes(args.summarize_hash_bytes)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the offload path shards per tensor-parallel rank with "
              "no exchange between ranks, so a rank's throughput is measured alone "
              "(use --gpus 1)", file=sys.stderr)
        sys.exit(2)
    other = {"agent_pool": run_agent_pool, "dense_scattered": run_dense_scattered,
             "layered_fp8": run_layered, "tiny": run_tiny, "load_cost": run_load_cost,
             "tp8_shard": run_tp8_shard, "hash": run_hash,
             "agent_pool_chunked": run_agent_pool_chunked, "plans": run_plans}
    if args.workload in other:
        out = other[args.workload](args)
        log(json.dumps(out))
        print(json.dumps(out), flush=True)
        return

    ctx = setup(args)
    N = ctx["N"]
    os.makedirs(os.path.dirname(args.detail), exist_ok=True)
    if args.isolated_only:
        iso = isolated(ctx)
        json.dump({"isolated": iso, "peak": ctx["peak"]}, open(args.detail, "w"), indent=1)
        ctx["tier"].close()
        ctx["cache"].close()
        return

    steps = run_steps(ctx, args)
    # the hash on its own, after the steps (before the isolated series, whose
    # last device copy calibrates the byte counters): the turn's prompt as one chain
    # (the step's serial part) and the batch case that the hash line's
    # roofline is taken on
    log("hash cases ...")
    hash_block = {"turn_56k_prompt": hash_case(ctx["torch"], [56000], 16),
                  "batch_65536x256": hash_case(ctx["torch"], [256] * 65536, 16)}
    hash_block["roofline"] = hash_roofline(hash_block["batch_65536x256"])
    for c in ("turn_56k_prompt", "batch_65536x256"):
        hash_block[c].pop("calls")
    log(f"hash: {hash_block}")
    iso = isolated(ctx)
    tier = ctx["tier"]
    plan_name = {N.EA_PLAN_DIRECT: "direct", N.EA_PLAN_STAGED: "staged"}
    plans = {"store": plan_name[tier.get_plan(N.EA_DIR_STORE)],
             "load": plan_name[tier.get_plan(N.EA_DIR_LOAD)]}
    log("restore-cost fit (Eq. 2) on one TP8 rank's shard ...")
    fit = restore_fit(ctx["peak"]["h2d"])
    log(f"restore fit: {fit['device']}")
    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle, one core) ...")
        cpu = cpu_baseline(ctx["W"], ctx["n_store"], ctx["n_load"], ctx["prefix"],
                           ctx["last_refill"])
        log(f"cpu baseline: {cpu}")
    tier.close()
    ctx["cache"].close()

    peak = ctx["peak"]
    traffic = committed_traffic() or {}
    # the dominant kernel of the step is the store (2,000 pages over the
    # link), timed in the step itself: it shares the link with the load
    roofline = {
        "bound": "host-link", "kernel": f"copy_host_link<store> ({plans['store']} plan, "
                                        f"2,000 pages, alongside the 1,500-page load)",
        "achieved": round(steps["store_gbs_in_step"], 2), "peak": round(peak["d2h"], 2),
        "peak_kind": "measured pinned hipMemcpyAsync device-to-host, 1 GiB, best of 10",
        "unit": "GB/s", "frac": round(steps["store_gbs_in_step"] / peak["d2h"], 4),
        "traffic": traffic.get("store"),
        # the counters see the store's HBM reads and its writes toward the
        # host: 2 x 2,000 pages of algorithmic bytes per launch
        "traffic_algorithmic": 2 * ctx["n_store"] * ctx["page"],
        "timing": f"HIP events on the store's stream around each of the {args.steps} timed "
                  f"launches",
        # the restore beside it, which has priority on the link (the store's
        # waves yield while it runs)
        "load_in_step": {"kernel": "copy_host_link<load> (1,500 pages, beside the store)",
                         "achieved": round(steps["load_gbs_in_step"], 2),
                         "peak": round(peak["h2d"], 2), "unit": "GB/s",
                         "frac": round(steps["load_gbs_in_step"] / peak["h2d"], 4)},
    }
    roofline_hbm = {
        "bound": "hbm", "kernel": "copy_hbm<gather> (paged gather of 2,000 pages to HBM)",
        "achieved": round(iso["gather_gbs"], 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
        "frac": round(iso["gather_gbs"] / HBM_PEAK_GBS, 4), "traffic": traffic.get("gather"),
        "traffic_algorithmic": 2 * ctx["n_store"] * ctx["page"],
        "scatter": {"achieved": round(iso["scatter_gbs"], 1),
                    "frac": round(iso["scatter_gbs"] / HBM_PEAK_GBS, 4),
                    "traffic": traffic.get("scatter"),
                    "traffic_algorithmic": 2 * ctx["n_store"] * ctx["page"]},
    }
    out = {
        "metric": "host-link GB/s for KV block store/load; HBM GB/s of paged gather/scatter",
        "value": round(steps["gbs"], 3), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(steps["ms"], 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u8", "data": "synthetic",
        "config": {"workload": "qwen3_30b_a3b_turn: store 2,000 + load 1,500 pages of 1.5 MiB, "
                               "hash the 56,000-token prompt as one chain, 20,000-page cache, "
                               "16 GiB tier",
                   "page_bytes": ctx["page"], "store_pages": ctx["n_store"],
                   "load_pages": ctx["n_load"], "plans": plans},
        "roofline": roofline, "roofline_hbm": roofline_hbm,
        "host_link": {"store_gbs": round(iso["store_gbs"], 2), "load_gbs": round(iso["load_gbs"], 2),
                      "store_gbs_in_step": round(steps["store_gbs_in_step"], 2),
                      "load_gbs_in_step": round(steps["load_gbs_in_step"], 2),
                      "peak_d2h": round(peak["d2h"], 2), "peak_h2d": round(peak["h2d"], 2),
                      "peak_bidir": round(peak["bidir"], 2),
                      "frac_store": round(iso["store_gbs"] / peak["d2h"], 4),
                      "frac_load": round(iso["load_gbs"] / peak["h2d"], 4),
                      "duplex_step_gbs": round(steps["gbs"], 2),
                      "frac_duplex_of_bidir": round(steps["gbs"] / peak["bidir"], 4)},
        "restore_fit": fit,
        "hash": hash_block,
        "cpu_baseline": cpu,
    }
    # launch order of each copy kernel in this run, for the profile summary:
    # the setup's prefix store, the warmup and timed steps, then the
    # isolated series (two untimed calls before each: a warm call and the
    # lead call right before the start event)
    # (then the restore fit's one store and its loads)
    dispatches = {
        "store": {"before": 1 + args.warmup, "timed": args.steps,
                  "after": 2 + 3 + 2 + N_ISO["store"] + 1},
        "load": {"before": args.warmup, "timed": args.steps,
                 "after": 2 + 3 + 2 + N_ISO["load"] + RESTORE_FIT_LOADS},
    }
    # hash calls of the turn itself (the set-up's prefix, warmup and timed
    # steps); the hash block's calls follow them
    dispatches["hash_calls_of_turn"] = 1 + args.warmup + args.steps
    json.dump({"line": out, "steps": steps, "isolated": iso, "peak": peak,
               "dispatches": dispatches, "argv": sys.argv[1:]}, open(args.detail, "w"),
              indent=1, default=float)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
