"""ctypes wrapper of the CPU oracle (oracle/libeao.so).

TEST INFRASTRUCTURE ONLY: the oracle is the plain single-threaded definition
of the KV-offload path (chained block keys, store, load, host-tier metadata
and write admission) that the GPU library is checked against.  Only the test
suite, the smoke check and the CPU-baseline leg of the benchmark use it.  It
imports nothing from the product package.

All arrays are numpy arrays in host memory.  Functions raise OracleError on a
negative status.
"""
import ctypes as C
import os

import numpy as np

from . import build as _build

_HERE = os.path.dirname(os.path.abspath(__file__))

EAO_OK, EAO_EINVAL, EAO_ENOMEM, EAO_ENOSPC, EAO_ENOTSUP = 0, -1, -2, -3, -5
SLOT_FREE, SLOT_PENDING, SLOT_RESIDENT = 0, 1, 2
ADMIT_CONDITIONED, ADMIT_ALWAYS, ADMIT_FIXED = 0, 1, 2


class OracleError(RuntimeError):
    def __init__(self, fn, code):
        super().__init__(f"{fn} returned {code}")
        self.code = code


class Shape(C.Structure):
    _fields_ = [("num_pages", C.c_int32), ("num_layers", C.c_int32),
                ("page_tokens", C.c_int32), ("num_kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("elem_bytes", C.c_int32),
                ("has_scales", C.c_int32), ("chunk_pages", C.c_int32)]


class Policy(C.Structure):
    _fields_ = [("theta_ppm", C.c_int64), ("kappa", C.c_int64),
                ("block_tokens", C.c_int64), ("beta_rank", C.c_int64),
                ("activity_window", C.c_int64), ("length_window", C.c_int32),
                ("mode", C.c_int32), ("telemetry", C.c_int32), ("_pad", C.c_int32)]


class Request(C.Structure):
    _fields_ = [("n_tokens", C.c_int64), ("h_tokens", C.c_int64),
                ("task_id", C.c_int64), ("now", C.c_int64),
                ("decided", C.c_int32), ("_pad", C.c_int32)]


class TierReport(C.Structure):
    _fields_ = [("time", C.c_int64), ("registered", C.c_int64),
                ("capacity_slots", C.c_int64), ("evictions", C.c_int64)]


class TierStats(C.Structure):
    _fields_ = [("capacity_slots", C.c_int64), ("allocated", C.c_int64),
                ("registered", C.c_int64), ("pinned", C.c_int64),
                ("evictions_total", C.c_int64), ("evictions_window", C.c_int64),
                ("clock", C.c_int64), ("active_tasks", C.c_int64),
                ("mean_prompt", C.c_double), ("working_set", C.c_double),
                ("last_pressure", C.c_int32), ("last_save", C.c_int32)]


_lib = None


def lib():
    """Load (building first if needed) the oracle shared library."""
    global _lib
    if _lib is None:
        path = _build.LIB
        if not os.path.exists(path):
            _build.build()
        L = C.CDLL(path)
        P, I32, I64, U8 = C.c_void_p, C.c_int32, C.c_int64, C.c_void_p
        sig = {
            "eao_sha256": (None, [P, C.c_uint64, P]),
            "eao_sha256_constants": (None, [P, P]),
            "eao_beta_rank": (I64, [I64, I64, I64, I64, I64]),
            "eao_working_set_bytes": (C.c_double, [C.c_double, C.c_double, C.c_double]),
            "eao_restore_time": (C.c_double, [C.c_double] * 4),
            "eao_obr": (C.c_double, [C.c_double] * 5),
            "eao_obr_limit": (C.c_double, [C.c_double] * 3),
            "eao_tier_chunks": (I64, [I64, I64, I64]),
            "eao_piece_bytes": (I64, [P]), "eao_page_bytes": (I64, [P]),
            "eao_trailer_bytes": (I64, [P]), "eao_slot_bytes": (I64, [P]),
            "eao_payload_bytes": (I64, [P]),
            "eao_cache_bytes": (I64, [P]), "eao_scale_bytes": (I64, [P]),
            "eao_hash_blocks": (C.c_int, [P, P, I32, I32, P, P, P]),
            "eao_store_blocks": (C.c_int, [P, P, P, P, I64, P, P, U8, I32]),
            "eao_load_blocks": (C.c_int, [P, P, I64, P, P, P, P, I32]),
            "eao_load_layer": (C.c_int, [P, P, I64, P, P, P, P, I32, I32]),
            "eao_layer_checksum": (C.c_int, [P, P, P, I32, P, I32, P]),
            "eao_tier_create": (C.c_int, [P, I64, P]),
            "eao_tier_destroy": (C.c_int, [P]),
            "eao_tier_capacity": (I64, [P]),
            "eao_tier_lookup": (C.c_int, [P, P, I64, P, P]),
            "eao_admission_fill": (C.c_int, [P, P, P, P, I64, P, P]),
            "eao_admission_fill_report": (C.c_int, [P, P, P, P, I64, P, I64, P, P]),
            "eao_tier_publish": (C.c_int, [P, I64, I64, P]),
            "eao_tier_alloc": (C.c_int, [P, P, P, I64, P, P]),
            "eao_tier_mark_stored": (C.c_int, [P, P, P, I64]),
            "eao_tier_unpin": (C.c_int, [P, P, I64]),
            "eao_tier_stats_get": (C.c_int, [P, P]),
            "eao_tier_export": (C.c_int, [P, P, P, P, P, P]),
            "eao_lru_reference": (C.c_int, [P, I64, P, I64, P]),
            "eao_lru_prefix_model": (C.c_int, [P, P, I64, P, I64, P]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def _check(fn, rc):
    if rc != EAO_OK:
        raise OracleError(fn, rc)


# ------------------------------------------------------------------ SHA-256

def sha256(data: bytes) -> bytes:
    buf = np.frombuffer(bytes(data), dtype=np.uint8) if len(data) else np.zeros(1, np.uint8)
    out = np.zeros(32, np.uint8)
    lib().eao_sha256(_ptr(buf), len(data), _ptr(out))
    return out.tobytes()


def sha256_constants():
    k = np.zeros(64, np.uint32)
    h0 = np.zeros(8, np.uint32)
    lib().eao_sha256_constants(_ptr(k), _ptr(h0))
    return k, h0


# ------------------------------------------------------- footprint, sizes

def beta_rank(layers, head_dim, elem_bytes, kv_heads, tp=1):
    return lib().eao_beta_rank(layers, head_dim, elem_bytes, kv_heads, tp)


def working_set_bytes(active_pool, mean_prompt_tokens, beta):
    return lib().eao_working_set_bytes(active_pool, mean_prompt_tokens, beta)


def tier_chunks(capacity_bytes, block_tokens, beta):
    return lib().eao_tier_chunks(capacity_bytes, block_tokens, beta)


def restore_time(n, beta, b_eff, tau):
    """Eq. 2: T_load(n) = n * beta / B_eff + tau."""
    return lib().eao_restore_time(n, beta, b_eff, tau)


def obr(n, beta, b_eff, tau, t_pf):
    """Eq. 2: OBR(n) = 1 - T_load(n) / (n * t_pf)."""
    return lib().eao_obr(n, beta, b_eff, tau, t_pf)


def obr_limit(beta, b_eff, t_pf):
    """OBR for long prefixes: 1 - beta / (B_eff * t_pf)."""
    return lib().eao_obr_limit(beta, b_eff, t_pf)


def make_shape(num_pages, num_layers, page_tokens, num_kv_heads, head_dim,
               elem_bytes, has_scales=False, chunk_pages=1):
    return Shape(num_pages, num_layers, page_tokens, num_kv_heads, head_dim,
                 elem_bytes, int(bool(has_scales)), chunk_pages)


def sizes(shape):
    L = lib()
    p = C.byref(shape)
    return dict(piece=L.eao_piece_bytes(p), page=L.eao_page_bytes(p),
                payload=L.eao_payload_bytes(p),
                trailer=L.eao_trailer_bytes(p), slot=L.eao_slot_bytes(p),
                cache=L.eao_cache_bytes(p), scales=L.eao_scale_bytes(p))


# ------------------------------------------------------------------ hashing

def hash_blocks(tokens, seq_offsets, block_tokens, parents=None):
    """Chained keys of every full block; returns (keys [K,32] u8, offsets)."""
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    seq_offsets = np.ascontiguousarray(seq_offsets, dtype=np.int64)
    n_seqs = len(seq_offsets) - 1
    lens = np.diff(seq_offsets)
    total = int(np.sum(lens // block_tokens)) if n_seqs > 0 and block_tokens > 0 else 0
    keys = np.zeros((max(total, 1), 32), np.uint8)
    offs = np.zeros(n_seqs + 1, np.int64)
    if parents is not None:
        parents = np.ascontiguousarray(parents, dtype=np.uint8).reshape(n_seqs, 32)
    rc = lib().eao_hash_blocks(_ptr(tokens) if tokens.size else None,
                               _ptr(seq_offsets), n_seqs, block_tokens,
                               _ptr(parents), _ptr(keys), _ptr(offs))
    _check("eao_hash_blocks", rc)
    return keys[:total], offs


# ------------------------------------------------------------------- copies

def _chunked(shape, pages, slots):
    if len(pages) != len(slots) * shape.chunk_pages:
        raise ValueError("need chunk_pages page ids per slot")


def store_blocks(shape, cache, scales, tier, block_ids, host_slots, mask=None):
    """block_ids: chunk_pages ids per entry of host_slots."""
    num_slots = tier.shape[0]
    block_ids = np.ascontiguousarray(block_ids, dtype=np.int32)
    host_slots = np.ascontiguousarray(host_slots, dtype=np.int64)
    _chunked(shape, block_ids, host_slots)
    if mask is not None:
        mask = np.ascontiguousarray(mask, dtype=np.uint8)
    rc = lib().eao_store_blocks(C.byref(shape), _ptr(cache), _ptr(scales),
                                _ptr(tier), num_slots, _ptr(block_ids),
                                _ptr(host_slots), _ptr(mask), len(host_slots))
    _check("eao_store_blocks", rc)


def load_blocks(shape, tier, cache, scales, host_slots, dst_pages):
    host_slots = np.ascontiguousarray(host_slots, dtype=np.int64)
    dst_pages = np.ascontiguousarray(dst_pages, dtype=np.int32)
    _chunked(shape, dst_pages, host_slots)
    rc = lib().eao_load_blocks(C.byref(shape), _ptr(tier), tier.shape[0],
                               _ptr(cache), _ptr(scales), _ptr(host_slots),
                               _ptr(dst_pages), len(host_slots))
    _check("eao_load_blocks", rc)


def load_layer(shape, tier, cache, scales, host_slots, dst_pages, layer):
    host_slots = np.ascontiguousarray(host_slots, dtype=np.int64)
    dst_pages = np.ascontiguousarray(dst_pages, dtype=np.int32)
    _chunked(shape, dst_pages, host_slots)
    rc = lib().eao_load_layer(C.byref(shape), _ptr(tier), tier.shape[0],
                              _ptr(cache), _ptr(scales), _ptr(host_slots),
                              _ptr(dst_pages), len(host_slots), layer)
    _check("eao_load_layer", rc)


def layer_checksum(shape, cache, scales, layer, pages):
    """uint64 [n]: XOR of the 64-bit words of each page's layer piece (and
    its scale word)."""
    pages = np.ascontiguousarray(pages, dtype=np.int32)
    out = np.zeros(max(len(pages), 1), np.uint64)
    rc = lib().eao_layer_checksum(C.byref(shape), _ptr(cache), _ptr(scales), layer,
                                  _ptr(pages), len(pages), _ptr(out))
    _check("eao_layer_checksum", rc)
    return out[:len(pages)]


# --------------------------------------------------------------------- tier

def make_policy(kappa, block_tokens, beta, theta_ppm=950000,
                activity_window=64, length_window=256, mode=ADMIT_CONDITIONED,
                telemetry=1):
    return Policy(theta_ppm, kappa, block_tokens, beta, activity_window,
                  length_window, mode, telemetry, 0)


class Tier:
    """Host-tier metadata of the oracle (no bytes: those live in arrays)."""

    def __init__(self, shape, capacity_bytes):
        self._h = C.c_void_p()
        _check("eao_tier_create",
               lib().eao_tier_create(C.byref(shape), capacity_bytes, C.byref(self._h)))
        self.capacity = lib().eao_tier_capacity(self._h)

    def close(self):
        if self._h:
            lib().eao_tier_destroy(self._h)
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def lookup(self, keys):
        keys = np.ascontiguousarray(keys, dtype=np.uint8).reshape(-1, 32)
        n = keys.shape[0]
        hit = C.c_int64()
        slots = np.full(max(n, 1), -1, np.int64)
        _check("eao_tier_lookup", lib().eao_tier_lookup(
            self._h, _ptr(keys) if n else None, n, C.byref(hit), _ptr(slots)))
        return hit.value, slots[:hit.value].copy()

    def admission(self, policy, n_tokens, h_tokens, task_id, now, keys, decided=-1):
        keys = np.ascontiguousarray(keys, dtype=np.uint8).reshape(-1, 32)
        n = keys.shape[0]
        req = Request(n_tokens, h_tokens, task_id, now, decided, 0)
        mask = np.zeros(max(n, 1), np.uint8)
        save = C.c_int32()
        _check("eao_admission_fill", lib().eao_admission_fill(
            self._h, C.byref(policy), C.byref(req), _ptr(keys) if n else None, n,
            _ptr(mask), C.byref(save)))
        return save.value, mask[:n].copy()

    def publish(self, now, window):
        """Telemetry report at time `now` (advances the tier's clock)."""
        rep = TierReport()
        _check("eao_tier_publish", lib().eao_tier_publish(self._h, now, window, C.byref(rep)))
        return rep

    def admission_report(self, policy, n_tokens, h_tokens, task_id, now, keys, report,
                         max_age, decided=-1):
        """Admission with the telemetry factor from `report` (a TierReport or
        None) when it is fresh."""
        keys = np.ascontiguousarray(keys, dtype=np.uint8).reshape(-1, 32)
        n = keys.shape[0]
        req = Request(n_tokens, h_tokens, task_id, now, decided, 0)
        mask = np.zeros(max(n, 1), np.uint8)
        save = C.c_int32()
        _check("eao_admission_fill_report", lib().eao_admission_fill_report(
            self._h, C.byref(policy), C.byref(req),
            None if report is None else C.byref(report), max_age,
            _ptr(keys) if n else None, n, _ptr(mask), C.byref(save)))
        return save.value, mask[:n].copy()

    def alloc(self, keys, mask=None):
        keys = np.ascontiguousarray(keys, dtype=np.uint8).reshape(-1, 32)
        n = keys.shape[0]
        if mask is not None:
            mask = np.ascontiguousarray(mask, dtype=np.uint8)
        slots = np.full(max(n, 1), -1, np.int64)
        count = C.c_int64()
        _check("eao_tier_alloc", lib().eao_tier_alloc(
            self._h, _ptr(keys) if n else None, _ptr(mask), n, _ptr(slots),
            C.byref(count)))
        return count.value, slots[:n].copy()

    def mark_stored(self, slots, mask=None):
        slots = np.ascontiguousarray(slots, dtype=np.int64)
        if mask is not None:
            mask = np.ascontiguousarray(mask, dtype=np.uint8)
        _check("eao_tier_mark_stored", lib().eao_tier_mark_stored(
            self._h, _ptr(slots), _ptr(mask), len(slots)))

    def unpin(self, slots):
        slots = np.ascontiguousarray(slots, dtype=np.int64)
        _check("eao_tier_unpin", lib().eao_tier_unpin(self._h, _ptr(slots), len(slots)))

    def stats(self):
        s = TierStats()
        _check("eao_tier_stats_get", lib().eao_tier_stats_get(self._h, C.byref(s)))
        return {f: getattr(s, f) for f, _ in TierStats._fields_}

    def export(self):
        K = self.capacity
        state = np.zeros(K, np.uint8)
        pins = np.zeros(K, np.int32)
        keys = np.zeros((K, 32), np.uint8)
        lru = np.zeros(K, np.int64)
        m = C.c_int64()
        _check("eao_tier_export", lib().eao_tier_export(
            self._h, _ptr(state), _ptr(pins), _ptr(keys), _ptr(lru), C.byref(m)))
        return dict(state=state, pins=pins, keys=keys, lru=lru[:m.value].copy())


# ------------------------------------------------- LRU reference model

def lru_reference(refs, capacity, declined=None):
    """Hits (uint8 [n]) of the reference model of the paper's appendix for
    one tier capacity in chunks.  refs: uint8 [n, 32] chunk keys in
    reference order; declined: optional bool/uint8 [n], misses to decline."""
    refs = np.ascontiguousarray(refs, dtype=np.uint8).reshape(-1, 32)
    n = len(refs)
    dec = None if declined is None else np.ascontiguousarray(declined, dtype=np.uint8)
    if dec is not None and len(dec) != n:
        raise ValueError("declined must have one entry per reference")
    hits = np.zeros(max(n, 1), np.uint8)
    _check("eao_lru_reference", lib().eao_lru_reference(
        _ptr(refs) if n else None, n, _ptr(dec) if n else None, int(capacity), _ptr(hits)))
    return hits[:n]


def lru_prefix_model(refs, req_off, capacity, declined=None):
    """Lookup hits per request (int64 [n_req]) under the host tier's own
    order; declined: optional bool [n_req], requests whose writes are
    skipped."""
    refs = np.ascontiguousarray(refs, dtype=np.uint8).reshape(-1, 32)
    offs = np.ascontiguousarray(req_off, dtype=np.int64)
    n_req = len(offs) - 1
    dec = None if declined is None else np.ascontiguousarray(declined, dtype=np.uint8)
    if dec is not None and len(dec) != n_req:
        raise ValueError("declined must have one entry per request")
    h = np.zeros(max(n_req, 1), np.int64)
    _check("eao_lru_prefix_model", lib().eao_lru_prefix_model(
        _ptr(refs) if len(refs) else None, _ptr(offs), n_req,
        _ptr(dec) if (dec is not None and n_req) else None, int(capacity), _ptr(h)))
    return h[:n_req]

