"""The C ABI library loads (without a GPU) and exports every entry point that
include/sae.h declares; the ctypes binding covers exactly that set."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared():
    txt = open(os.path.join(ROOT, "include", "sae.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(sae_[a-z_0-9]+)\s*\(", txt)))


@pytest.fixture(scope="module")
def lib():
    from paper_2605_18825_amd import _lib, build
    if not os.path.exists(_lib.LIB_PATH):
        build.build()
    return ctypes.CDLL(_lib.LIB_PATH)


def test_header_declares_the_hot_calls():
    d = declared()
    for name in ("sae_prefix_match", "sae_score_select", "sae_feedback_update"):
        assert name in d


def test_library_exports_every_declared_symbol(lib):
    missing = [n for n in declared() if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_matches_header():
    from paper_2605_18825_amd import _lib
    assert _lib.exported_symbols() == declared()


def test_status_strings(lib):
    lib.sae_status_str.restype = ctypes.c_char_p
    assert lib.sae_status_str(0) == b"ok"
    assert lib.sae_status_str(-1) == b"invalid argument"


def test_create_rejects_bad_config_without_gpu(lib):
    """Validation runs on the host before any device call."""
    from paper_2605_18825_amd._lib import SaeConfig, load
    L = load()
    cfg = SaeConfig()
    cfg.n_instances = 1
    cfg.blocks_per_instance = 1024
    cfg.n_queues = 9
    cfg.max_k = 64
    out = ctypes.c_void_p()
    assert L.sae_create(ctypes.byref(cfg), ctypes.byref(out)) == -1
    assert b"n_queues" in L.sae_last_error(None)
    cfg.n_queues = 2
    cfg.queue_kind[0] = 0
    cfg.queue_kind[1] = 0
    assert L.sae_create(ctypes.byref(cfg), ctypes.byref(out)) == -1
    assert b"evict-first" in L.sae_last_error(None)
    cfg.queue_kind[1] = 2
    cfg.max_requests = -1
    assert L.sae_create(ctypes.byref(cfg), ctypes.byref(out)) == -1
    assert b"max_requests" in L.sae_last_error(None)
    cfg.max_requests = 0
    cfg.max_k = 0
    assert L.sae_create(ctypes.byref(cfg), ctypes.byref(out)) == -1


def test_hot_calls_reject_null_context(lib):
    from paper_2605_18825_amd._lib import load
    L = load()
    assert L.sae_score_select(None, 0, 1, None, 0, None, None, None, None, None, None) == -1
    assert L.sae_prefix_match(None, 1, 1, None, None, None, 0, 0, None, None, None) == -1
    assert L.sae_match_select(None, 1, 1, None, None, None, 0, 0, None, None, 0, 1, None, 0, None, None, None, None,
                              None, None) == -1
    assert L.sae_feedback_update(None, 0, None) == -1
    n = ctypes.c_int32()
    assert L.sae_get_intervals(None, 0, 0, None, 0, ctypes.byref(n), None) == -1
