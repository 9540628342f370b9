"""Python binding of libsae with the C ABI's names.

Argument marshalling only: every operation runs in the HIP library.  Device
buffers are torch tensors on the current HIP device; the stream is torch's
current stream unless one is passed.
"""
import ctypes

import torch

from . import _lib
from ._lib import IVL_CAP, N_BINS, SaeConfig, SaeCounters, SaeError, SaeParams, SaePool, SaePredictor  # noqa: F401

KIND_EVICT_FIRST, KIND_STRUCTURAL, KIND_LOGNORMAL, KIND_RECENCY = 0, 1, 2, 3
META_VALID, META_LEAF, META_REF = 0x40, 0x80, 0x100
PM_TOUCH, PM_STATS, PM_INTERVALS = 1, 2, 4
SS_COMMIT, SS_ENGINE_SCAN, SS_ENGINE_BATCHED, SS_FORCE_FALLBACK, SS_CASCADE = 1, 2, 4, 8, 16
FB_FORCE = 1
HINT_DECODE, HINT_UNTEMPLATED, HINT_MULTI_TURN, HINT_AGENTIC, HINT_CONVERSATION, HINT_SHARED_PREFIX = 1, 2, 4, 8, 16, 32
ROLE_EVICT, ROLE_STRUCT, ROLE_CHAT, ROLE_AGENT = 0, 1, 2, 3
LEARN_TOKEN_WEIGHTS, LEARN_QUEUE_WEIGHTS, LEARN_LOGNORMAL, LEARN_DECAY_POWER = 1, 2, 4, 8
LEARN_TOKEN_EMA, LEARN_QUEUE_REL = 16, 32
# the paper's initial token weights (system, user, tool, response, cot), Sec. 5
PAPER_INIT_W = (2.0, 1.5, 1.0, 1.0, 0.1)
ST_NAMES = {1: "INDEX_FULL", 2: "GHOST_FULL", 4: "BAD_OFFSET", 8: "FUTURE_ACCESS",
            16: "SLOT_BUSY", 32: "SELECT_FALLBACK", 64: "BAD_BLOCK", 128: "BAD_HASH"}


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise SaeError("expected a device tensor")
    if not t.is_contiguous():
        raise SaeError("expected a contiguous tensor")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _check(ctx, st):
    if st != 0:
        L = _lib.load()
        msg = L.sae_last_error(ctx).decode()
        raise SaeError("%s: %s" % (L.sae_status_str(st).decode(), msg))


# --------------------------------------------------------------------- layout
def pack_meta(queue, tau, ntok, valid=True, leaf=True, ref=False):
    """uint16 meta (as int32 tensor values): queue | tau<<3 | flags | (ntok-1)<<9."""
    m = (queue.to(torch.int32) & 7) | ((tau.to(torch.int32) & 7) << 3) | (((ntok.to(torch.int32) - 1) & 15) << 9)

    def flag(v, bit):
        if isinstance(v, torch.Tensor):
            return v.to(torch.int32) * bit
        return bit if v else 0
    return m | flag(valid, META_VALID) | flag(leaf, META_LEAF) | flag(ref, META_REF)


def meta_to_u16(m):
    """int32 values in [0, 65535] -> int16 tensor holding the same bits."""
    return (m.to(torch.int32) & 0xFFFF).to(torch.int16)


def unpack_meta(meta16):
    m = meta16.to(torch.int32) & 0xFFFF
    return dict(queue=m & 7, tau=(m >> 3) & 7, valid=(m & META_VALID) != 0, leaf=(m & META_LEAF) != 0,
                ref=(m & META_REF) != 0, ntok=((m >> 9) & 15) + 1)


def pack_off(ob, omax):
    return ((omax.to(torch.int64) << 16) | (ob.to(torch.int64) & 0xFFFF)).to(torch.int64)


def off_to_u32(off):
    """int64 values in [0, 2^32) -> int32 tensor holding the same bits."""
    return (off - ((off >= 2 ** 31).to(torch.int64) << 32)).to(torch.int32)


# ----------------------------------------------------------------- the C ABI
def sae_create(n_instances, blocks_per_instance, queue_kinds, max_k, ghost_window=0, index_log2=0, max_requests=0):
    L = _lib.load()
    cfg = SaeConfig()
    cfg.n_instances = n_instances
    cfg.blocks_per_instance = blocks_per_instance
    cfg.n_queues = len(queue_kinds)
    for i, k in enumerate(queue_kinds):
        cfg.queue_kind[i] = int(k)
    cfg.max_k = max_k
    cfg.ghost_window = ghost_window
    cfg.index_log2 = index_log2
    cfg.max_requests = max_requests
    out = ctypes.c_void_p()
    st = L.sae_create(ctypes.byref(cfg), ctypes.byref(out))
    if st != 0:
        raise SaeError("sae_create: %s: %s" % (L.sae_status_str(st).decode(), L.sae_last_error(None).decode()))
    return out


def sae_destroy(ctx):
    _check(ctx, _lib.load().sae_destroy(ctx))


def sae_bind_pool(ctx, last_access, meta, off, hash, parent, child_count, ref_count, access_count):
    p = SaePool()
    for name, t in (("last_access", last_access), ("meta", meta), ("off", off), ("hash", hash),
                    ("parent", parent), ("child_count", child_count), ("ref_count", ref_count),
                    ("access_count", access_count)):
        setattr(p, name, _ptr(t).value)
    _check(ctx, _lib.load().sae_bind_pool(ctx, ctypes.byref(p)))


def make_params(n_queues, w=1.0, alpha=1.0, mu=0.0, sigma=1.0, gamma=1.0, eta=0.01, temperature=1.0,
                beta=0.1, K=32, learn=LEARN_TOKEN_WEIGHTS | LEARN_QUEUE_WEIGHTS, beta_ln=0.1):
    p = SaeParams()

    def fill(arr, v, n):
        vals = list(v) if hasattr(v, "__len__") else [v] * n
        for i in range(len(arr)):
            arr[i] = float(vals[i]) if i < len(vals) else (1.0 if arr is p.sigma else 0.0)
    fill(p.w, w, 5)
    fill(p.alpha, alpha, n_queues)
    fill(p.mu, mu, n_queues)
    fill(p.sigma, sigma, n_queues)
    for i in range(n_queues, 8):
        p.alpha[i] = 1.0
        p.sigma[i] = 1.0
    p.gamma, p.eta, p.temperature, p.beta, p.beta_ln = gamma, eta, temperature, beta, beta_ln
    p.K, p.learn = int(K), int(learn)
    return p


def sae_set_params(ctx, inst, params, stream=None):
    _check(ctx, _lib.load().sae_set_params(ctx, inst, ctypes.byref(params), _stream(stream)))


def sae_get_params(ctx, inst, stream=None):
    p = SaeParams()
    _check(ctx, _lib.load().sae_get_params(ctx, inst, ctypes.byref(p), _stream(stream)))
    return p


def sae_get_counters(ctx, inst, stream=None):
    c = SaeCounters()
    _check(ctx, _lib.load().sae_get_counters(ctx, inst, ctypes.byref(c), _stream(stream)))
    return c


def sae_set_counters(ctx, inst, counters, stream=None):
    _check(ctx, _lib.load().sae_set_counters(ctx, inst, ctypes.byref(counters), _stream(stream)))


def sae_block_type(counts_u8, tau_u8, stream=None):
    n = counts_u8.shape[0]
    _check(None, _lib.load().sae_block_type(_ptr(counts_u8), n, _ptr(tau_u8), _stream(stream)))


FN_LN, FN_EXP, FN_ERFC = 0, 1, 2


def sae_recipe_eval(fn, x_f32, y_f32, stream=None):
    """The device realisation of ln / exp / erfc of the fp32 recipe, element-wise."""
    _check(None, _lib.load().sae_recipe_eval(int(fn), x_f32.numel(), _ptr(x_f32), _ptr(y_f32), _stream(stream)))


def sae_classify_blocks(ctx, hint_u8, meta_u16, roles, stream=None):
    """Algorithm 1 Classify on the device: rewrites the queue bits of meta."""
    r = (ctypes.c_int32 * 4)(*[int(x) for x in roles])
    _check(ctx, _lib.load().sae_classify_blocks(ctx, hint_u8.numel(), _ptr(hint_u8), _ptr(meta_u16), r,
                                                _stream(stream)))


def sae_index_build(ctx, stream=None):
    _check(ctx, _lib.load().sae_index_build(ctx, _stream(stream)))


def sae_insert_blocks(ctx, ids, hash, parent, last_access, meta, off, inst=None, stream=None):
    n = ids.numel()
    _check(ctx, _lib.load().sae_insert_blocks(ctx, n, _ptr(inst), _ptr(ids), _ptr(hash), _ptr(parent),
                                              _ptr(last_access), _ptr(meta), _ptr(off), _stream(stream)))


def sae_ref_blocks(ctx, ids, delta, inst=None, stream=None):
    _check(ctx, _lib.load().sae_ref_blocks(ctx, ids.numel(), _ptr(inst), _ptr(ids), int(delta), _stream(stream)))


def sae_prefix_match(ctx, hashes, lens, now, flags, match_len, matched_ids=None, inst=None, stream=None):
    n_req, max_len = hashes.shape
    _check(ctx, _lib.load().sae_prefix_match(ctx, n_req, max_len, _ptr(hashes), _ptr(lens), _ptr(inst), int(now),
                                             int(flags), _ptr(match_len), _ptr(matched_ids), _stream(stream)))


def sae_score_select(ctx, now, k, flags, victims, count, decision, decision_count, scores=None, k_per_inst=None,
                     stream=None):
    _check(ctx, _lib.load().sae_score_select(ctx, int(now), int(k), _ptr(k_per_inst), int(flags), _ptr(victims),
                                             _ptr(scores), _ptr(count), _ptr(decision), _ptr(decision_count),
                                             _stream(stream)))


def sae_match_select(ctx, hashes, lens, pm_now, pm_flags, match_len, now, k, flags, victims, count, decision,
                     decision_count, matched_ids=None, inst=None, scores=None, k_per_inst=None, stream=None):
    """sae_prefix_match then sae_score_select, as one call (same results)."""
    n_req, max_len = hashes.shape
    _check(ctx, _lib.load().sae_match_select(ctx, n_req, max_len, _ptr(hashes), _ptr(lens), _ptr(inst), int(pm_now),
                                             int(pm_flags), _ptr(match_len), _ptr(matched_ids), int(now), int(k),
                                             _ptr(k_per_inst), int(flags), _ptr(victims), _ptr(scores), _ptr(count),
                                             _ptr(decision), _ptr(decision_count), _stream(stream)))


def sae_feedback_update(ctx, flags=0, stream=None):
    _check(ctx, _lib.load().sae_feedback_update(ctx, int(flags), _stream(stream)))


def sae_poll_status(ctx, stream=None):
    b = ctypes.c_uint32()
    _check(ctx, _lib.load().sae_poll_status(ctx, _stream(stream), ctypes.byref(b)))
    return b.value


def sae_select_stats(ctx, inst, n_queues, stream=None):
    buf = (ctypes.c_uint32 * (4 * n_queues))()
    _check(ctx, _lib.load().sae_select_stats(ctx, inst, ctypes.cast(buf, ctypes.c_void_p), _stream(stream)))
    return [tuple(buf[4 * q:4 * q + 4]) for q in range(n_queues)]


def sae_profile_enable(ctx, enable=True):
    _check(ctx, _lib.load().sae_profile_enable(ctx, 1 if enable else 0))


def sae_profile_read(ctx):
    ms = ctypes.c_double()
    n = ctypes.c_int64()
    _check(ctx, _lib.load().sae_profile_read(ctx, ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def sae_state_size(ctx):
    n = ctypes.c_size_t()
    _check(ctx, _lib.load().sae_state_size(ctx, ctypes.byref(n)))
    return n.value


def sae_save_state(ctx, inst, stream=None):
    """Instance `inst`'s context-held state as bytes (see include/sae.h)."""
    n = sae_state_size(ctx)
    buf = ctypes.create_string_buffer(n)
    _check(ctx, _lib.load().sae_save_state(ctx, inst, ctypes.cast(buf, ctypes.c_void_p), n, _stream(stream)))
    return buf.raw


def sae_load_state(ctx, inst, blob, stream=None):
    buf = ctypes.create_string_buffer(bytes(blob), len(blob))
    _check(ctx, _lib.load().sae_load_state(ctx, inst, ctypes.cast(buf, ctypes.c_void_p), len(blob),
                                           _stream(stream)))


def sae_get_intervals(ctx, inst, queue, cap=IVL_CAP, stream=None):
    """Algorithm 4's interval buffer of (inst, queue), oldest first (host list)."""
    buf = (ctypes.c_int32 * max(cap, 1))()
    n = ctypes.c_int32()
    _check(ctx, _lib.load().sae_get_intervals(ctx, inst, queue, ctypes.cast(buf, ctypes.c_void_p), cap,
                                              ctypes.byref(n), _stream(stream)))
    return list(buf[:min(n.value, cap)])


def sae_predict_sessions(h_bf16, w, work, logit, pred=None, stream=None):
    """Session predictor (Sec. 3.3) on n hidden states: h_bf16 is an int16
    tensor [n][d] of bf16 bit patterns; w holds device tensors w1 (int16
    [256][d], bf16 bits), b1, w2 [64][256], b2, w3 [64], b3 [1] (float32)."""
    n, d = h_bf16.shape
    p = SaePredictor()
    for name in ("w1", "b1", "w2", "b2", "w3", "b3"):
        setattr(p, name, _ptr(w[name]).value)
    _check(None, _lib.load().sae_predict_sessions(n, d, _ptr(h_bf16), ctypes.byref(p), _ptr(work), _ptr(logit),
                                                  _ptr(pred), _stream(stream)))


PRED_NOALLOC_MAX_N = 4096


def sae_predict_sessions_noalloc(h_bf16, w, logit, pred=None, stream=None):
    """As sae_predict_sessions, with the library's own per-GPU buffer in place
    of `work` (n <= PRED_NOALLOC_MAX_N); allocates nothing."""
    n, d = h_bf16.shape
    p = SaePredictor()
    for name in ("w1", "b1", "w2", "b2", "w3", "b3"):
        setattr(p, name, _ptr(w[name]).value)
    _check(None, _lib.load().sae_predict_sessions_noalloc(n, d, _ptr(h_bf16), ctypes.byref(p), _ptr(logit),
                                                          _ptr(pred), _stream(stream)))


def status_names(bits):
    return [v for k, v in ST_NAMES.items() if bits & k]
