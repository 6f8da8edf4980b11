"""ctypes declarations of libea.so (include/ea.h).

Argument marshalling only: every step of the offload path runs inside the
HIP library.  Loading fails loudly when libea.so has not been built; there is
no fallback.  torch is imported first so that the library binds to the HIP
runtime torch already loaded (both carry the soname libamdhip64.so.7), which
keeps torch's streams and device pointers valid inside the library.
"""
import ctypes as C
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
# EA_LIB_PATH selects another build of the same library (e.g. for A/B timing)
LIB_PATH = os.environ.get("EA_LIB_PATH") or os.path.join(_PKG, "libea.so")

EA_OK, EA_EINVAL, EA_ENOMEM, EA_ENOSPC, EA_EHIP, EA_ENOTSUP = 0, -1, -2, -3, -4, -5
EA_ADMIT_CONDITIONED, EA_ADMIT_ALWAYS, EA_ADMIT_FIXED = 0, 1, 2
EA_PLAN_AUTO, EA_PLAN_DIRECT, EA_PLAN_STAGED = 0, 1, 2
EA_DIR_STORE, EA_DIR_LOAD, EA_DIR_BOTH = 0, 1, 2
EA_SLOT_FREE, EA_SLOT_PENDING, EA_SLOT_RESIDENT = 0, 1, 2


class CacheDesc(C.Structure):
    _fields_ = [("base", C.c_void_p), ("scale_base", C.c_void_p),
                ("num_pages", C.c_int32), ("num_layers", C.c_int32),
                ("page_tokens", C.c_int32), ("num_kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("elem_bytes", C.c_int32)]


class TierInfo(C.Structure):
    _fields_ = [("capacity_slots", C.c_int64), ("slot_bytes", C.c_int64),
                ("piece_bytes", C.c_int64), ("page_bytes", C.c_int64),
                ("trailer_bytes", C.c_int64), ("capacity_bytes", C.c_int64),
                ("host_base", C.c_void_p), ("device_base", C.c_void_p),
                ("chunk_pages", C.c_int64)]


class Policy(C.Structure):
    _fields_ = [("theta_ppm", C.c_int64), ("kappa", C.c_int64),
                ("block_tokens", C.c_int64), ("beta_rank", C.c_int64),
                ("activity_window", C.c_int64), ("length_window", C.c_int32),
                ("mode", C.c_int32), ("telemetry", C.c_int32), ("_pad", C.c_int32)]


class Request(C.Structure):
    _fields_ = [("n_tokens", C.c_int64), ("h_tokens", C.c_int64),
                ("task_id", C.c_int64), ("now", C.c_int64),
                ("decided", C.c_int32), ("_pad", C.c_int32)]


class TierStats(C.Structure):
    _fields_ = [("capacity_slots", C.c_int64), ("allocated", C.c_int64),
                ("registered", C.c_int64), ("pinned", C.c_int64),
                ("evictions_total", C.c_int64), ("evictions_window", C.c_int64),
                ("clock", C.c_int64), ("active_tasks", C.c_int64),
                ("mean_prompt", C.c_double), ("working_set", C.c_double),
                ("last_pressure", C.c_int32), ("last_save", C.c_int32),
                ("bytes_stored", C.c_int64), ("bytes_loaded", C.c_int64),
                ("store_calls", C.c_int64), ("load_calls", C.c_int64)]


class TierReport(C.Structure):
    _fields_ = [("time", C.c_int64), ("registered", C.c_int64),
                ("capacity_slots", C.c_int64), ("evictions", C.c_int64)]


class ControllerConfig(C.Structure):
    _fields_ = [("report_interval", C.c_int64), ("read_interval", C.c_int64),
                ("max_report_age", C.c_int64), ("window", C.c_int64),
                ("manual_clock", C.c_int32), ("_pad", C.c_int32)]


class ControllerStatus(C.Structure):
    _fields_ = [("now", C.c_int64), ("reports_published", C.c_int64),
                ("published", TierReport), ("seen", TierReport),
                ("have_seen", C.c_int32), ("fresh", C.c_int32),
                ("decisions", C.c_int64), ("skips", C.c_int64),
                ("fresh_decisions", C.c_int64)]


_P, _I32, _I64, _INT = C.c_void_p, C.c_int32, C.c_int64, C.c_int

SIGNATURES = {
    "ea_strerror": (C.c_char_p, [_INT]),
    "ea_last_hip_error": (_INT, []),
    "ea_cache_create": (_INT, [_P, _P]),
    "ea_cache_destroy": (_INT, [_P]),
    "ea_tier_create": (_INT, [_P, _I64, _INT, _P]),
    "ea_tier_create_chunked": (_INT, [_P, _I32, _I64, _INT, _P]),
    "ea_tier_destroy": (_INT, [_P]),
    "ea_tier_get_info": (_INT, [_P, _P]),
    "ea_hash_blocks": (_INT, [_P, _P, _I32, _I32, _P, _P, _P, _P]),
    "ea_hash_blocks_device": (_INT, [_P, _I64, _P, _I32, _I32, _P, _P, _I64, _P, _P]),
    "ea_hash_blocks_device_offsets": (_INT, [_P, _I64, _P, _I32, _I32, _P, _P, _I64, _P, _P]),
    "ea_hash_blocks_device_offsets_noalloc": (_INT, [_P, _I64, _P, _I32, _I32, _P, _P, _I64, _P,
                                                     _P]),
    "ea_tier_lookup": (_INT, [_P, _P, _I64, _P, _P]),
    "ea_admission_fill": (_INT, [_P, _P, _P, _P, _I64, _P, _P]),
    "ea_admission_fill_report": (_INT, [_P, _P, _P, _P, _I64, _P, _I64, _P, _P]),
    "ea_tier_publish": (_INT, [_P, _I64, _I64, _P]),
    "ea_controller_create": (_INT, [_P, _P, _P, _P]),
    "ea_controller_destroy": (_INT, [_P]),
    "ea_controller_advance": (_INT, [_P, _I64]),
    "ea_controller_decide": (_INT, [_P, _I64, _I64, _I64, _I32, _P, _I64, _P, _P]),
    "ea_controller_get_status": (_INT, [_P, _P]),
    "ea_tier_alloc": (_INT, [_P, _P, _P, _I64, _P, _P]),
    "ea_tier_unpin": (_INT, [_P, _P, _I64]),
    "ea_tier_stats": (_INT, [_P, _P]),
    "ea_tier_export": (_INT, [_P, _P, _P, _P, _P, _P]),
    "ea_store_blocks": (_INT, [_P, _P, _P, _P, _P, _I32, _P]),
    "ea_load_blocks": (_INT, [_P, _P, _P, _P, _I32, _P]),
    "ea_load_blocks_layered": (_INT, [_P, _P, _P, _P, _I32, _P, _P, _I32]),
    "ea_gather_blocks": (_INT, [_P, _P, _I32, _P, _I64, _P]),
    "ea_scatter_blocks": (_INT, [_P, _P, _I64, _P, _I32, _P]),
    "ea_layer_checksum": (_INT, [_P, _I32, _P, _I32, _P, _I64, _P]),
    "ea_tier_set_plan": (_INT, [_P, _INT, _INT]),
    "ea_tier_get_plan": (_INT, [_P, _INT, _P]),
    "ea_peak_probe": (_INT, [_P, _P, _I64, _INT, _INT, _P]),
    "ea_reuse_distances": (_INT, [_P, _I64, _P, _P]),
    "ea_prefix_coverage": (_INT, [_P, _P, _I64, _P, _I64, _P]),
    "ea_lru_simulate": (_INT, [_P, _I64, _P, _I64, _P]),
    "ea_lru_simulate_prefix": (_INT, [_P, _P, _I64, _P, _I64, _P]),
}

_lib = None


def load():
    """Load libea.so (bound to torch's HIP runtime when torch is present)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build the HIP library first "
            "(python -c 'import __graft_entry__ as g; g.build()')")
    try:
        import torch  # noqa: F401  (binds libamdhip64.so.7 to torch's copy)
    except ImportError:
        pass
    lib = C.CDLL(LIB_PATH, mode=C.RTLD_GLOBAL)
    for name, (res, args) in SIGNATURES.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


class EAError(RuntimeError):
    def __init__(self, fn, code):
        lib = load()
        text = lib.ea_strerror(code).decode()
        hip = lib.ea_last_hip_error() if code == EA_EHIP else 0
        super().__init__(f"{fn}: {text} ({code})" + (f", hip error {hip}" if hip else ""))
        self.code = code
        self.hip_error = hip


def check(fn, rc):
    if rc != EA_OK:
        raise EAError(fn, rc)
    return rc
