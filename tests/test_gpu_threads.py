"""Several host threads share one cache and one tier.

The tier and the hash workspace are internally locked, so callers may share
them across threads.  Here four copy threads store and load their own slots
and pages on their own streams, in batches that travel both in the kernel
arguments (up to 32 entries) and through the index ring.  At the same time
a request thread hashes, looks up, admits, allocates, stores and unpins on
its own slots, and a hash thread computes keys.  Every thread's results, and
the final cache and tier images, must equal the oracle's replay of each
thread's operations (their slots and destination pages are disjoint and no
source page is ever written, so any interleaving gives the same end state).
"""
import threading

import numpy as np
import pytest

import oracle
from paper_2609_33762_amd import _native as N, api
from paper_2609_33762_amd import workloads as W

from gpu_common import Pair, need_gpu

pytestmark = pytest.mark.gpu

B = 16


def test_threads_share_one_cache_and_tier():
    torch = need_gpu()
    n_copy = 4
    P, S = 512, 512
    p = Pair(P, 2, B, 2, 64, 2, S, seed=31)  # 8 KiB pieces, 16 KiB slots
    r = W.rng(31)
    perm = r.permutation(P).astype(np.int32)
    src_of = [perm[64 * i:64 * (i + 1)] for i in range(n_copy)]
    dst_of = [perm[256 + 48 * i:256 + 48 * (i + 1)] for i in range(n_copy)]
    req_src = perm[448:512]
    slots_of = [np.arange(128 + 96 * i, 128 + 96 * (i + 1), dtype=np.int64) for i in range(n_copy)]
    errors, ops = [], [[] for _ in range(n_copy)]
    streams = [torch.cuda.Stream() for _ in range(n_copy + 1)]

    def copier(i):
        try:
            rr = W.rng(500 + i)
            for _ in range(12):
                n = int(rr.integers(1, 97))
                sl = rr.choice(slots_of[i], n, replace=False)
                src = rr.choice(src_of[i], n)
                p.tier.store(p.cache, src, sl, stream=streams[i])
                ops[i].append(("store", src, sl))
                m = int(rr.integers(1, min(n, 48) + 1))
                ls = rr.choice(sl, m, replace=False)
                dst = rr.choice(dst_of[i], m, replace=False)
                p.tier.load(p.cache, ls, dst, stream=streams[i])
                ops[i].append(("load", ls, dst))
        except Exception as e:  # reported by the main thread
            errors.append(e)

    pol = api.make_policy(kappa=0, block_tokens=B, beta_rank=1024, mode=N.EA_ADMIT_ALWAYS)
    agent = W.tokens(77, B * 24)
    lengths = [B * 4, B * 8 + 5, B * 8 + 9, B * 16, B * 12, B * 24]
    req_log = []

    def requester():
        try:
            rr = W.rng(600)
            for t, n_tok in enumerate(lengths):
                toks = agent[:n_tok]
                keys, _ = api.hash_blocks(toks, np.array([0, n_tok]), B)
                h, hs = p.tier.lookup(keys)
                save, mask = p.tier.admission(pol, n_tok, B * h, 0, t, keys)
                cnt, sl = p.tier.alloc(keys, mask)
                got = sl >= 0
                src = rr.choice(req_src, int(got.sum()))
                if got.any():
                    p.tier.store(p.cache, src, sl[got], stream=streams[n_copy])
                    p.tier.unpin(sl[got])
                if h:
                    p.tier.unpin(hs)
                req_log.append((keys, h, hs, save, mask, sl, src))
        except Exception as e:
            errors.append(e)

    hash_ok = []

    def hasher():
        try:
            rr = W.rng(700)
            for _ in range(30):
                lens = [int(x) for x in rr.integers(0, 600, size=int(rr.integers(1, 6)))]
                toks, offs = W.sequences(int(rr.integers(0, 1 << 30)), lens)
                got, goff = api.hash_blocks(toks, offs, B)
                want, woff = oracle.hash_blocks(toks, offs, B)
                hash_ok.append(np.array_equal(got, want) and np.array_equal(goff, woff))
        except Exception as e:
            errors.append(e)

    threads = [threading.Thread(target=copier, args=(i,)) for i in range(n_copy)]
    threads += [threading.Thread(target=requester), threading.Thread(target=hasher)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    torch.cuda.synchronize()
    assert not errors, errors
    assert len(hash_ok) == 30 and all(hash_ok)

    # the request thread against the oracle's tier, request by request
    ot = oracle.Tier(p.oshape, S * p.sizes["slot"])
    opol = oracle.make_policy(kappa=0, block_tokens=B, beta=1024, mode=oracle.ADMIT_ALWAYS)
    for t, (keys, h, hs, save, mask, sl, src) in enumerate(req_log):
        okeys, _ = oracle.hash_blocks(agent[:lengths[t]], np.array([0, lengths[t]]), B)
        assert np.array_equal(keys, okeys), t
        oh, ohs = ot.lookup(keys)
        assert oh == h and np.array_equal(ohs, hs), t
        osave, omask = ot.admission(opol, lengths[t], B * h, 0, t, keys)
        assert osave == save and np.array_equal(omask, mask), t
        _, osl = ot.alloc(keys, omask)
        assert np.array_equal(osl, sl), t
        got = osl >= 0
        if got.any():
            ot.mark_stored(osl[got])
            ot.unpin(osl[got])
            p.o_store(src, osl[got])
        if oh:
            ot.unpin(ohs)
    assert req_log[-1][1] == max(lengths[:-1]) // B  # the last request hit its stored prefix
    a, b = p.tier.export(), ot.export()
    for k in ("state", "pins", "keys", "lru"):
        assert np.array_equal(a[k], b[k]), k

    # the copy threads' operations, thread by thread
    for i in range(n_copy):
        for kind, x, y in ops[i]:
            if kind == "store":
                p.o_store(x, y)
            else:
                p.o_load(x, y)
    p.assert_equal("threads")
    p.close()


def test_hashing_on_two_streams_runs_concurrently():
    # Hash buffers are kept per (device, stream) and no lock is held across
    # a wait for the GPU, so two threads hashing on two streams do not queue
    # behind each other.  Each thread hashes a 3,500-key chain (one serial
    # chain takes milliseconds and occupies one compute unit), synchronously
    # and asynchronously; keys equal the oracle's, and the two threads
    # together take well under twice one thread's time.
    import time
    torch = need_gpu()
    n = 56000
    seqs = [W.sequences(800 + i, [n]) for i in range(2)]
    want = [oracle.hash_blocks(t, o, B)[0] for t, o in seqs]
    streams = [torch.cuda.Stream() for _ in range(2)]
    d_toks = [torch.as_tensor(t, device="cuda") for t, _ in seqs]
    outs = [torch.zeros((n // B, 32), dtype=torch.uint8, device="cuda") for _ in range(2)]
    got, errors = [None, None], []

    def work(i, reps):
        try:
            for _ in range(reps):
                got[i], _ = api.hash_blocks(seqs[i][0], seqs[i][1], B, stream=streams[i])
                api.hash_blocks_device(d_toks[i], seqs[i][1], B, outs[i], stream=streams[i])
                streams[i].synchronize()
        except Exception as e:
            errors.append(e)

    work(0, 1)  # warm up both paths and the workspace of stream 0
    work(1, 1)
    t0 = time.perf_counter()
    work(0, 3)
    alone = time.perf_counter() - t0
    threads = [threading.Thread(target=work, args=(i, 3)) for i in range(2)]
    t0 = time.perf_counter()
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    both = time.perf_counter() - t0
    assert not errors, errors
    for i in range(2):
        assert np.array_equal(got[i], want[i]), i
        assert np.array_equal(outs[i].cpu().numpy(), want[i]), i
    print(f"one thread {alone * 1e3:.1f} ms, two threads {both * 1e3:.1f} ms")
    assert both < 1.5 * alone, (alone, both)
