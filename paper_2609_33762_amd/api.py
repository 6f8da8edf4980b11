"""Python binding of libea: thin wrappers that pass torch device pointers,
numpy host arrays and HIP stream handles to the C ABI (include/ea.h).

Nothing here computes any part of the offload path; it marshals arguments
and raises EAError on a negative status.
"""
import ctypes as C

import numpy as np

from . import _native as N
from ._native import EAError  # noqa: F401


def _ptr(a):
    return None if a is None else a.ctypes.data


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _i64(a):
    return np.ascontiguousarray(a, dtype=np.int64)


def _u8(a):
    return np.ascontiguousarray(a, dtype=np.uint8)


def _nbytes(t):
    return t.numel() * t.element_size()


def _check_offsets(offs, n_tokens):
    if len(offs) < 1:
        raise ValueError("seq_offsets needs at least one entry")
    if len(offs) > 1 and (offs[0] < 0 or (np.diff(offs) < 0).any()):
        raise ValueError("seq_offsets must be non-decreasing from >= 0")
    if offs[-1] > n_tokens:
        raise ValueError(f"seq_offsets end at {offs[-1]}, past the {n_tokens} tokens given")


def current_stream():
    import torch
    return torch.cuda.current_stream().cuda_stream


def _stream(s):
    if s is None:
        return current_stream()
    if isinstance(s, int):
        return s
    return s.cuda_stream


class Cache:
    """A caller-owned paged KV cache: `kv` is a CUDA tensor holding
    [L][P][2][T][H][D] elements of elem_bytes each (any dtype, contiguous);
    `scales` an optional contiguous CUDA float32 tensor [L][P][2]."""

    def __init__(self, kv, num_pages, num_layers, page_tokens, num_kv_heads,
                 head_dim, elem_bytes, scales=None):
        lib = N.load()
        assert kv.is_cuda and kv.is_contiguous()
        piece = 2 * page_tokens * num_kv_heads * head_dim * elem_bytes
        if kv.numel() * kv.element_size() < num_layers * num_pages * piece:
            raise ValueError("kv tensor is smaller than the described cache")
        if scales is not None:
            assert scales.is_cuda and scales.is_contiguous()
            if scales.numel() * scales.element_size() < num_layers * num_pages * 8:
                raise ValueError("scale tensor is smaller than [L][P][2] float32")
        self.kv, self.scales = kv, scales
        self.desc = N.CacheDesc(kv.data_ptr(), scales.data_ptr() if scales is not None else None,
                                num_pages, num_layers, page_tokens, num_kv_heads,
                                head_dim, elem_bytes)
        self.num_pages, self.num_layers = num_pages, num_layers
        self.piece_bytes = piece
        # one page per slot: the layers' pieces, then the scale trailer
        trailer = (num_layers * 8 + 255) // 256 * 256 if scales is not None else 0
        self.slot_bytes = num_layers * piece + trailer
        self._h = C.c_void_p()
        N.check("ea_cache_create", lib.ea_cache_create(C.byref(self.desc), C.byref(self._h)))

    @property
    def handle(self):
        return self._h

    def close(self):
        if self._h:
            N.load().ea_cache_destroy(self._h)
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _slots_fit(self, buf, n, what):
        if not buf.is_cuda:
            raise ValueError(f"{what} must be a device tensor")
        if _nbytes(buf) < n * self.slot_bytes:
            raise ValueError(f"{what} holds {_nbytes(buf)} bytes, {n} slots need "
                             f"{n * self.slot_bytes}")

    def gather(self, block_ids, dst, stream=None):
        ids = _i32(block_ids)
        self._slots_fit(dst, len(ids), "dst")
        N.check("ea_gather_blocks", N.load().ea_gather_blocks(
            self._h, _ptr(ids), len(ids), dst.data_ptr(), _nbytes(dst), _stream(stream)))

    def scatter(self, src, dst_pages, stream=None):
        d = _i32(dst_pages)
        self._slots_fit(src, len(d), "src")
        N.check("ea_scatter_blocks", N.load().ea_scatter_blocks(
            self._h, src.data_ptr(), _nbytes(src), _ptr(d), len(d), _stream(stream)))

    def layer_checksum(self, layer, pages, d_out, stream=None):
        """d_out (device uint64 tensor, >= len(pages) entries) gets the XOR
        checksum of each page's piece of `layer` (and its scale word)."""
        import torch
        p = _i32(pages)
        if not d_out.is_cuda or d_out.dtype not in (torch.int64, torch.uint64) or \
                not d_out.is_contiguous() or d_out.numel() < len(p):
            raise ValueError("d_out must be a contiguous 64-bit device tensor of len(pages)")
        N.check("ea_layer_checksum", N.load().ea_layer_checksum(
            self._h, layer, _ptr(p), len(p), d_out.data_ptr(), d_out.numel(), _stream(stream)))


def make_policy(kappa, block_tokens, beta_rank, theta_ppm=950000, activity_window=64,
                length_window=256, mode=N.EA_ADMIT_CONDITIONED, telemetry=1):
    return N.Policy(theta_ppm, kappa, block_tokens, beta_rank, activity_window,
                    length_window, mode, telemetry, 0)


class Tier:
    """Library-owned pinned host tier shaped like `cache`, one key per slot of
    chunk_pages pages."""

    def __init__(self, cache, capacity_bytes, numa_node=-1, chunk_pages=1):
        lib = N.load()
        self._h = C.c_void_p()
        N.check("ea_tier_create_chunked", lib.ea_tier_create_chunked(
            cache.handle, chunk_pages, capacity_bytes, numa_node, C.byref(self._h)))
        info = N.TierInfo()
        N.check("ea_tier_get_info", lib.ea_tier_get_info(self._h, C.byref(info)))
        self.info = {f: getattr(info, f) for f, _ in N.TierInfo._fields_}
        self.capacity = info.capacity_slots
        self.slot_bytes = info.slot_bytes
        self.chunk_pages = info.chunk_pages

    def close(self):
        """Free the tier; raises EAError (and keeps it) while a Controller is
        attached to it."""
        if self._h:
            N.check("ea_tier_destroy", N.load().ea_tier_destroy(self._h))
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            # a controller collected in the same cycle still holds it: that
            # controller frees the tier when it closes
            self._orphaned = True

    def host_view(self):
        """numpy uint8 [K_H, slot_bytes] view of the pinned slots (no copy)."""
        n = self.capacity * self.slot_bytes
        buf = (C.c_uint8 * n).from_address(self.info["host_base"])
        return np.frombuffer(buf, dtype=np.uint8).reshape(self.capacity, self.slot_bytes)

    # -------------------------------------------------- metadata / policy
    def lookup(self, keys):
        keys = _u8(keys).reshape(-1, 32)
        n = keys.shape[0]
        hit = C.c_int64()
        slots = np.full(max(n, 1), -1, np.int64)
        N.check("ea_tier_lookup", N.load().ea_tier_lookup(
            self._h, _ptr(keys) if n else None, n, C.byref(hit), _ptr(slots)))
        return hit.value, slots[:hit.value].copy()

    def admission(self, policy, n_tokens, h_tokens, task_id, now, keys, decided=-1):
        keys = _u8(keys).reshape(-1, 32)
        n = keys.shape[0]
        req = N.Request(n_tokens, h_tokens, task_id, now, decided, 0)
        mask = np.zeros(max(n, 1), np.uint8)
        save = C.c_int32()
        N.check("ea_admission_fill", N.load().ea_admission_fill(
            self._h, C.byref(policy), C.byref(req), _ptr(keys) if n else None, n,
            _ptr(mask), C.byref(save)))
        return save.value, mask[:n].copy()

    def publish(self, now, window):
        """The tier's telemetry report at time `now` (N.TierReport)."""
        rep = N.TierReport()
        N.check("ea_tier_publish", N.load().ea_tier_publish(self._h, now, window, C.byref(rep)))
        return rep

    def admission_report(self, policy, n_tokens, h_tokens, task_id, now, keys, report,
                         max_age, decided=-1):
        """Admission with the telemetry factor from `report` (N.TierReport or
        None) when it is fresh."""
        keys = _u8(keys).reshape(-1, 32)
        n = keys.shape[0]
        req = N.Request(n_tokens, h_tokens, task_id, now, decided, 0)
        mask = np.zeros(max(n, 1), np.uint8)
        save = C.c_int32()
        N.check("ea_admission_fill_report", N.load().ea_admission_fill_report(
            self._h, C.byref(policy), C.byref(req),
            None if report is None else C.byref(report), max_age,
            _ptr(keys) if n else None, n, _ptr(mask), C.byref(save)))
        return save.value, mask[:n].copy()

    def alloc(self, keys, mask=None):
        keys = _u8(keys).reshape(-1, 32)
        n = keys.shape[0]
        mask = None if mask is None else _u8(mask)
        slots = np.full(max(n, 1), -1, np.int64)
        count = C.c_int64()
        N.check("ea_tier_alloc", N.load().ea_tier_alloc(
            self._h, _ptr(keys) if n else None, _ptr(mask), n, _ptr(slots), C.byref(count)))
        return count.value, slots[:n].copy()

    def unpin(self, slots):
        slots = _i64(slots)
        N.check("ea_tier_unpin", N.load().ea_tier_unpin(self._h, _ptr(slots), len(slots)))

    def stats(self):
        s = N.TierStats()
        N.check("ea_tier_stats", N.load().ea_tier_stats(self._h, C.byref(s)))
        return {f: getattr(s, f) for f, _ in N.TierStats._fields_}

    def export(self):
        K = self.capacity
        state = np.zeros(K, np.uint8)
        pins = np.zeros(K, np.int32)
        keys = np.zeros((K, 32), np.uint8)
        lru = np.zeros(K, np.int64)
        m = C.c_int64()
        N.check("ea_tier_export", N.load().ea_tier_export(
            self._h, _ptr(state), _ptr(pins), _ptr(keys), _ptr(lru), C.byref(m)))
        return dict(state=state, pins=pins, keys=keys, lru=lru[:m.value].copy())

    def set_plan(self, direction, plan):
        N.check("ea_tier_set_plan", N.load().ea_tier_set_plan(self._h, direction, plan))

    def get_plan(self, direction):
        p = C.c_int()
        N.check("ea_tier_get_plan", N.load().ea_tier_get_plan(self._h, direction, C.byref(p)))
        return p.value

    # -------------------------------------------------------------- copies
    def _pages_per_slot(self, pages, slots):
        if len(pages) != len(slots) * self.chunk_pages:
            raise ValueError("need chunk_pages page ids per slot")

    def store(self, cache, block_ids, host_slots, mask=None, stream=None):
        """block_ids: chunk_pages page ids per entry of host_slots."""
        ids, slots = _i32(block_ids), _i64(host_slots)
        self._pages_per_slot(ids, slots)
        mask = None if mask is None else _u8(mask)
        N.check("ea_store_blocks", N.load().ea_store_blocks(
            cache.handle, self._h, _ptr(ids), _ptr(slots), _ptr(mask), len(slots),
            _stream(stream)))

    def load(self, cache, host_slots, dst_pages, stream=None):
        slots, dst = _i64(host_slots), _i32(dst_pages)
        self._pages_per_slot(dst, slots)
        N.check("ea_load_blocks", N.load().ea_load_blocks(
            self._h, cache.handle, _ptr(slots), _ptr(dst), len(slots), _stream(stream)))

    def load_layered(self, cache, host_slots, dst_pages, copy_stream, layer_events):
        """layer_events: torch.cuda.Event objects, one per layer."""
        slots, dst = _i64(host_slots), _i32(dst_pages)
        self._pages_per_slot(dst, slots)
        if len(layer_events) != cache.num_layers:
            raise ValueError(f"need one event per layer ({cache.num_layers}), "
                             f"got {len(layer_events)}")
        for e in layer_events:
            if not e.cuda_event:  # torch creates the HIP event at its first record
                e.record(copy_stream)
        evs = (C.c_void_p * len(layer_events))(*[e.cuda_event for e in layer_events])
        N.check("ea_load_blocks_layered", N.load().ea_load_blocks_layered(
            self._h, cache.handle, _ptr(slots), _ptr(dst), len(slots),
            _stream(copy_stream), evs, len(layer_events)))

    def peak_probe(self, dev_buf, nbytes, direction, reps=10):
        g = C.c_double()
        N.check("ea_peak_probe", N.load().ea_peak_probe(
            self._h, dev_buf.data_ptr(), nbytes, direction, reps, C.byref(g)))
        return g.value


def hash_blocks(tokens, seq_offsets, block_tokens, parents=None, stream=None):
    """Chained keys of every full block, computed on the GPU.  Host in, host
    out; returns (keys uint8 [K, 32], key_offsets int64 [n_seqs + 1])."""
    tokens, offs = _i32(tokens), _i64(seq_offsets)
    _check_offsets(offs, len(tokens))
    n_seqs = len(offs) - 1
    total = int(np.sum(np.diff(offs) // block_tokens)) if n_seqs > 0 and block_tokens > 0 else 0
    keys = np.zeros((max(total, 1), 32), np.uint8)
    koffs = np.zeros(n_seqs + 1, np.int64)
    if parents is not None and _u8(parents).size != 32 * n_seqs:
        raise ValueError("parents must hold 32 bytes per sequence")
    par = None if parents is None else _u8(parents).reshape(n_seqs, 32)
    N.check("ea_hash_blocks", N.load().ea_hash_blocks(
        _ptr(tokens) if tokens.size else None, _ptr(offs), n_seqs, block_tokens,
        _ptr(par), _ptr(keys), _ptr(koffs), _stream(stream)))
    return keys[:total], koffs


def hash_blocks_device(d_tokens, seq_offsets, block_tokens, d_keys_out, d_parents=None,
                       stream=None):
    """Asynchronous variant on device tensors; returns key_offsets."""
    offs = _i64(seq_offsets)
    _check_device_buffers(d_tokens, d_keys_out, d_parents, len(offs) - 1)
    _check_offsets(offs, d_tokens.numel())
    n_seqs = len(offs) - 1
    total = int(np.sum(np.diff(offs) // block_tokens)) if n_seqs > 0 and block_tokens > 0 else 0
    if _nbytes(d_keys_out) < 32 * total:
        raise ValueError(f"d_keys_out holds {_nbytes(d_keys_out)} bytes, {total} keys need "
                         f"{32 * total}")
    koffs = np.empty(n_seqs + 1, np.int64)
    N.check("ea_hash_blocks_device", N.load().ea_hash_blocks_device(
        d_tokens.data_ptr(), d_tokens.numel(), _ptr(offs), n_seqs, block_tokens,
        None if d_parents is None else d_parents.data_ptr(), d_keys_out.data_ptr(),
        _nbytes(d_keys_out) // 32, _ptr(koffs), _stream(stream)))
    return koffs


def hash_blocks_device_offsets(d_tokens, d_seq_offsets, block_tokens, d_keys_out,
                               d_key_offsets_out, d_parents=None, stream=None, noalloc=False):
    """Fully asynchronous variant: sequence offsets (int64 [n_seqs + 1]) and
    key offsets (int64 [n_seqs + 1]) are device tensors too; on the device,
    malformed offsets or too many keys leave d_key_offsets_out[0] = -1.
    noalloc=True calls the entry point that allocates nothing (fixed device
    memory per device; calls must not overlap on one device)."""
    import torch
    n_seqs = d_seq_offsets.numel() - 1
    _check_device_buffers(d_tokens, d_keys_out, d_parents, n_seqs)
    for t, what in ((d_seq_offsets, "d_seq_offsets"), (d_key_offsets_out, "d_key_offsets_out")):
        if not t.is_cuda or t.dtype != torch.int64 or not t.is_contiguous():
            raise ValueError(f"{what} must be a contiguous int64 device tensor")
    if n_seqs < 0 or d_key_offsets_out.numel() < n_seqs + 1:
        raise ValueError("need n_seqs + 1 entries in both offset tensors")
    name = "ea_hash_blocks_device_offsets" + ("_noalloc" if noalloc else "")
    N.check(name, getattr(N.load(), name)(
        d_tokens.data_ptr(), d_tokens.numel(), d_seq_offsets.data_ptr(), n_seqs, block_tokens,
        None if d_parents is None else d_parents.data_ptr(), d_keys_out.data_ptr(),
        _nbytes(d_keys_out) // 32, d_key_offsets_out.data_ptr(), _stream(stream)))


def _check_device_buffers(d_tokens, d_keys_out, d_parents, n_seqs):
    import torch
    if not (d_tokens.is_cuda and d_keys_out.is_cuda):
        raise ValueError("tokens and keys must be device tensors")
    if d_tokens.dtype != torch.int32 or not d_tokens.is_contiguous():
        raise ValueError("d_tokens must be a contiguous int32 tensor")
    if not d_keys_out.is_contiguous():
        raise ValueError("d_keys_out must be contiguous")
    if d_parents is not None and (not d_parents.is_cuda or _nbytes(d_parents) < 32 * n_seqs):
        raise ValueError("d_parents must be a device tensor of 32 bytes per sequence")


# ------------------------------------------- reuse-distance capacity tool

def reuse_distances(refs):
    """(prev_dist, next_dist), int64 [n] each, of a chunk reference stream
    (uint8 [n, 32] keys in reference order); -1 marks a first or last
    reference.  Host-only."""
    refs = _u8(refs).reshape(-1, 32)
    n = len(refs)
    prev = np.zeros(max(n, 1), np.int64)
    nxt = np.zeros(max(n, 1), np.int64)
    N.check("ea_reuse_distances", N.load().ea_reuse_distances(
        _ptr(refs) if n else None, n, _ptr(prev), _ptr(nxt)))
    return prev[:n], nxt[:n]


def prefix_coverage(prev_dist, req_off, caps):
    """int64 [n_requests, n_caps]: leading hits of each request in an LRU
    tier of caps[c] chunks that admits every miss.  Host-only."""
    prev, offs, caps = _i64(prev_dist), _i64(req_off), _i64(caps)
    n_req, n_caps = len(offs) - 1, len(caps)
    if n_req < 0:
        raise ValueError("req_off needs at least one entry")
    if offs[-1] > len(prev):
        raise ValueError("req_off runs past the distance array")
    out = np.zeros((max(n_req, 1), max(n_caps, 1)), np.int64)
    N.check("ea_prefix_coverage", N.load().ea_prefix_coverage(
        _ptr(prev) if len(prev) else None, _ptr(offs), n_req,
        _ptr(caps) if n_caps else None, n_caps, _ptr(out)))
    return out[:n_req, :n_caps]


def lru_simulate(refs, capacity, declined=None):
    """uint8 [n] hits of the reference model in an LRU tier of `capacity`
    chunks, misses at `declined` references left out.  Host-only."""
    refs = _u8(refs).reshape(-1, 32)
    n = len(refs)
    dec = None if declined is None else _u8(declined)
    if dec is not None and len(dec) != n:
        raise ValueError("declined must have one entry per reference")
    hits = np.zeros(max(n, 1), np.uint8)
    N.check("ea_lru_simulate", N.load().ea_lru_simulate(
        _ptr(refs) if n else None, n, _ptr(dec) if (dec is not None and n) else None,
        int(capacity), _ptr(hits)))
    return hits[:n]


def lru_simulate_prefix(refs, req_off, capacity, declined=None):
    """int64 [n_requests] lookup hits under the host tier's own order;
    declined: optional bool [n_requests].  Host-only."""
    refs = _u8(refs).reshape(-1, 32)
    offs = _i64(req_off)
    n_req = len(offs) - 1
    dec = None if declined is None else _u8(declined)
    if dec is not None and len(dec) != n_req:
        raise ValueError("declined must have one entry per request")
    out = np.zeros(max(n_req, 1), np.int64)
    N.check("ea_lru_simulate_prefix", N.load().ea_lru_simulate_prefix(
        _ptr(refs) if len(refs) else None, _ptr(offs), n_req,
        _ptr(dec) if (dec is not None and n_req) else None, int(capacity), _ptr(out)))
    return out[:n_req]


# ------------------------------------------------- wall-clock controller

class Controller:
    """Write-admission controller on a tier: reports every report_interval,
    scheduler reads every read_interval, fresh for max_report_age, windows
    of `window` (all microseconds; the paper's 1 s, 0.5 s, 5 s and 60 s by
    default).  manual_clock=True: no thread, advance() moves the clock."""

    def __init__(self, tier, policy, report_interval=1_000_000, read_interval=500_000,
                 max_report_age=5_000_000, window=60_000_000, manual_clock=False):
        self._h = C.c_void_p()
        cfg = N.ControllerConfig(report_interval, read_interval, max_report_age, window,
                                 int(bool(manual_clock)), 0)
        N.check("ea_controller_create", N.load().ea_controller_create(
            tier._h, C.byref(policy), C.byref(cfg), C.byref(self._h)))
        self._tier = tier  # the tier outlives its controllers

    def close(self):
        if self._h:
            N.load().ea_controller_destroy(self._h)
            self._h = C.c_void_p()
            if getattr(self._tier, "_orphaned", False):
                self._tier.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def advance(self, now):
        N.check("ea_controller_advance", N.load().ea_controller_advance(self._h, now))

    def decide(self, n_tokens, h_tokens, task_id, keys, decided=-1):
        keys = _u8(keys).reshape(-1, 32)
        n = keys.shape[0]
        mask = np.zeros(max(n, 1), np.uint8)
        save = C.c_int32()
        N.check("ea_controller_decide", N.load().ea_controller_decide(
            self._h, n_tokens, h_tokens, task_id, decided, _ptr(keys) if n else None, n,
            _ptr(mask), C.byref(save)))
        return save.value, mask[:n].copy()

    def status(self):
        st = N.ControllerStatus()
        N.check("ea_controller_get_status", N.load().ea_controller_get_status(
            self._h, C.byref(st)))
        rep = lambda r: {f: getattr(r, f) for f, _ in N.TierReport._fields_}  # noqa: E731
        out = {f: getattr(st, f) for f, _ in N.ControllerStatus._fields_}
        out["published"], out["seen"] = rep(st.published), rep(st.seen)
        return out

