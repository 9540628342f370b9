"""ctypes declarations of libsae's C ABI (include/sae.h).

Loading fails loudly when the HIP library has not been built: there is no
CPU fallback for any call.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsae.so")

MAX_QUEUES = 8
N_TYPES = 5
N_BINS = 8
IVL_CAP = 4096


class SaeConfig(ctypes.Structure):
    _fields_ = [
        ("n_instances", ctypes.c_int32),
        ("blocks_per_instance", ctypes.c_int32),
        ("n_queues", ctypes.c_int32),
        ("queue_kind", ctypes.c_int32 * MAX_QUEUES),
        ("max_k", ctypes.c_int32),
        ("ghost_window", ctypes.c_int32),
        ("index_log2", ctypes.c_int32),
        ("max_requests", ctypes.c_int32),
    ]


class SaeParams(ctypes.Structure):
    _fields_ = [
        ("w", ctypes.c_float * N_TYPES),
        ("alpha", ctypes.c_float * MAX_QUEUES),
        ("mu", ctypes.c_float * MAX_QUEUES),
        ("sigma", ctypes.c_float * MAX_QUEUES),
        ("gamma", ctypes.c_float),
        ("eta", ctypes.c_float),
        ("temperature", ctypes.c_float),
        ("beta", ctypes.c_float),
        ("beta_ln", ctypes.c_float),
        ("K", ctypes.c_int32),
        ("learn", ctypes.c_uint32),
    ]


class SaeCounters(ctypes.Structure):
    _fields_ = [
        ("evicted", ctypes.c_int32 * N_TYPES),
        ("missed", ctypes.c_int32 * N_TYPES),
        ("hits", ctypes.c_int32 * MAX_QUEUES),
        ("evictions", ctypes.c_int32 * MAX_QUEUES),
        ("eviction_count", ctypes.c_int64),
        ("pending", ctypes.c_int32),
        ("n_updates", ctypes.c_int32),
        ("bin_hits", ctypes.c_int32 * N_BINS),
        ("bin_missed", ctypes.c_int32 * N_BINS),
        ("type_hits", ctypes.c_int32 * N_TYPES),
        ("type_added", ctypes.c_int32 * N_TYPES),
        ("resident", ctypes.c_int32 * MAX_QUEUES),
    ]


class SaePredictor(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("w1", "b1", "w2", "b2", "w3", "b3")]


class SaePool(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "last_access", "meta", "off", "hash", "parent", "child_count", "ref_count", "access_count")]


# exported symbol -> (restype, argtypes)
_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_U32 = ctypes.c_uint32
_I64 = ctypes.c_int64
SIGNATURES = {
    "sae_status_str": (ctypes.c_char_p, [_I32]),
    "sae_last_error": (ctypes.c_char_p, [_P]),
    "sae_create": (_I32, [ctypes.POINTER(SaeConfig), ctypes.POINTER(_P)]),
    "sae_destroy": (_I32, [_P]),
    "sae_bind_pool": (_I32, [_P, ctypes.POINTER(SaePool)]),
    "sae_set_params": (_I32, [_P, _I32, ctypes.POINTER(SaeParams), _P]),
    "sae_get_params": (_I32, [_P, _I32, ctypes.POINTER(SaeParams), _P]),
    "sae_get_counters": (_I32, [_P, _I32, ctypes.POINTER(SaeCounters), _P]),
    "sae_set_counters": (_I32, [_P, _I32, ctypes.POINTER(SaeCounters), _P]),
    "sae_block_type": (_I32, [_P, _I64, _P, _P]),
    "sae_recipe_eval": (_I32, [_I32, _I64, _P, _P, _P]),
    "sae_classify_blocks": (_I32, [_P, _I32, _P, _P, ctypes.POINTER(_I32), _P]),
    "sae_index_build": (_I32, [_P, _P]),
    "sae_insert_blocks": (_I32, [_P, _I32, _P, _P, _P, _P, _P, _P, _P, _P]),
    "sae_ref_blocks": (_I32, [_P, _I32, _P, _P, _I32, _P]),
    "sae_prefix_match": (_I32, [_P, _I32, _I32, _P, _P, _P, _I32, _U32, _P, _P, _P]),
    "sae_score_select": (_I32, [_P, _I32, _I32, _P, _U32, _P, _P, _P, _P, _P, _P]),
    "sae_match_select": (_I32, [_P, _I32, _I32, _P, _P, _P, _I32, _U32, _P, _P, _I32, _I32, _P, _U32, _P, _P, _P, _P,
                                _P, _P]),
    "sae_feedback_update": (_I32, [_P, _U32, _P]),
    "sae_poll_status": (_I32, [_P, _P, ctypes.POINTER(_U32)]),
    "sae_get_intervals": (_I32, [_P, _I32, _I32, _P, _I32, ctypes.POINTER(_I32), _P]),
    "sae_state_size": (_I32, [_P, ctypes.POINTER(ctypes.c_size_t)]),
    "sae_save_state": (_I32, [_P, _I32, _P, ctypes.c_size_t, _P]),
    "sae_load_state": (_I32, [_P, _I32, _P, ctypes.c_size_t, _P]),
    "sae_predict_sessions": (_I32, [_I32, _I32, _P, ctypes.POINTER(SaePredictor), _P, _P, _P, _P]),
    "sae_predict_sessions_noalloc": (_I32, [_I32, _I32, _P, ctypes.POINTER(SaePredictor), _P, _P, _P]),
    "sae_select_stats": (_I32, [_P, _I32, _P, _P]),
    "sae_profile_enable": (_I32, [_P, _I32]),
    "sae_profile_read": (_I32, [_P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_I64)]),
}

_lib = None


class SaeError(RuntimeError):
    pass


def load():
    """Load libsae.so; raise if it is missing (never fall back)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise SaeError("libsae.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def exported_symbols():
    return sorted(SIGNATURES)
