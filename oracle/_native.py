"""TEST INFRASTRUCTURE — loader for the oracle's C scoring recipe (oracle/dsr.c).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may use the
oracle.  The library is built with gcc (never hipcc) and shares no code with the
HIP path.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dsr.c")
_SRC_RL = os.path.join(_HERE, "recency.c")  # the recency-list selection (a second CPU baseline)
_LIB = os.path.join(_HERE, "liboracle_dsr.so")

# -ffp-contract=off: no fused multiply-add unless written as fmaf();
# no -ffast-math: IEEE binary32 semantics, subnormals kept.
CFLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared", "-std=c99"]


def build(force=True):
    """Compile dsr.c and recency.c into liboracle_dsr.so with gcc."""
    if not force and os.path.exists(_LIB):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", *CFLAGS, "-o", tmp, _SRC, _SRC_RL, "-lm"])
    os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < max(os.path.getmtime(_SRC),
                                                                   os.path.getmtime(_SRC_RL)):
            build()
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i64, i32, f32 = ctypes.c_int64, ctypes.c_int32, ctypes.c_float
        for name in ("oracle_ln", "oracle_exp", "oracle_erfc", "oracle_inv_sigma_sqrt2"):
            fn = getattr(L, name)
            fn.argtypes = [f32]
            fn.restype = f32
        L.oracle_pow01.argtypes = [f32, f32]
        L.oracle_pow01.restype = f32
        L.oracle_p_lognormal.argtypes = [i32, f32, f32]
        L.oracle_p_lognormal.restype = f32
        L.oracle_p_structural.argtypes = [i32, i32, f32]
        L.oracle_p_structural.restype = f32
        L.oracle_score_blocks.argtypes = [i64, i32] + [P] * 6 + [P] * 5 + [f32, P, P]
        L.oracle_score_blocks.restype = None
        for name in ("oracle_ln_v", "oracle_exp_v", "oracle_erfc_v"):
            getattr(L, name).argtypes = [i64, P, P]
        L.oracle_pow01_v.argtypes = [i64, P, f32, P]
        L.oracle_p_lognormal_v.argtypes = [i64, P, f32, f32, P]
        L.oracle_p_structural_v.argtypes = [i64, P, P, f32, P]
        L.oracle_rl_select.argtypes = [i32, i32, i32, i32, f32, f32, P, P, P, P, P, P, P, P]
        L.oracle_rl_select.restype = i32
        L.oracle_struct_select.argtypes = [i32, i32, f32, P, i64, P, P, P, P, P, P, P, P]
        L.oracle_struct_select.restype = i32
        _lib = L
    return _lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _f32(x):
    return np.ascontiguousarray(x, dtype=np.float32)


def _i32(x):
    return np.ascontiguousarray(x, dtype=np.int32)


def ln(x):
    x = _f32(x)
    y = np.empty_like(x)
    lib().oracle_ln_v(x.size, _ptr(x), _ptr(y))
    return y


def exp(x):
    x = _f32(x)
    y = np.empty_like(x)
    lib().oracle_exp_v(x.size, _ptr(x), _ptr(y))
    return y


def erfc(x):
    x = _f32(x)
    y = np.empty_like(x)
    lib().oracle_erfc_v(x.size, _ptr(x), _ptr(y))
    return y


def pow01(r, gamma):
    r = _f32(r)
    y = np.empty_like(r)
    lib().oracle_pow01_v(r.size, _ptr(r), float(gamma), _ptr(y))
    return y


def p_lognormal(dt, mu, sigma):
    dt = _i32(dt)
    y = np.empty(dt.shape, np.float32)
    lib().oracle_p_lognormal_v(dt.size, _ptr(dt), float(mu), float(sigma), _ptr(y))
    return y


def p_structural(ob, omax, gamma):
    ob = _i32(ob)
    omax = _i32(omax)
    y = np.empty(ob.shape, np.float32)
    lib().oracle_p_structural_v(ob.size, _ptr(ob), _ptr(omax), float(gamma), _ptr(y))
    return y


def score_blocks(now, last_access, queue, tau, ntok, ob, omax, kind, alpha, mu, sigma, w, gamma):
    """Per-block selection key (uint32 bits of P, or of float(num_tokens) for an
    evict-first queue) and local priority p, via the C recipe."""
    la, q, t, nt, o1, o2 = (_i32(a) for a in (last_access, queue, tau, ntok, ob, omax))
    kd = _i32(np.resize(np.asarray(kind, np.int32), 8))
    al, m, s = (_f32(np.resize(np.asarray(a, np.float32), 8)) for a in (alpha, mu, sigma))
    ww = _f32(w)
    n = la.size
    key = np.empty(n, np.uint32)
    p = np.empty(n, np.float32)
    lib().oracle_score_blocks(n, int(now), _ptr(la), _ptr(q), _ptr(t), _ptr(nt), _ptr(o1), _ptr(o2),
                              _ptr(kd), _ptr(al), _ptr(m), _ptr(s), _ptr(ww), float(gamma),
                              _ptr(key), _ptr(p))
    return key, p
