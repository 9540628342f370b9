"""Seeded request traces shaped like the paper's single-/multi-turn workloads.

The paper's trace-driven evaluation mixes five request categories (Table 2):
chat and agent sessions are multi-turn, tool use, programming and document QA
requests are single-turn.  Requests are injected at a fixed interval (the
paper sweeps 0.02 - 0.08 s; 30 ms here).  This generator stands in for those
traces; no record of any dataset is reproduced.

Recipe (every draw from one PCG64 stream per trace, in request order):

* slot s is served at time t0 + s * interval_ms and its category is drawn
  from Table 2's mix.  For a multi-turn category, the earliest turn of that
  category that is due by then is served; if none is due (and always for a
  single-turn category) a new session of that category starts.  The request
  mix therefore follows Table 2 from the first request on;
* turns of a multi-turn session: Geometric with mean 6; the gap before the
  next turn is log-normal with Table 3's parameters (chat mu 4.82 s, sigma
  1.25; agent mu 2.28 s, sigma 1.34);
* every request starts with a system prompt from a pool of 2,000 templates
  drawn Zipf(1.1) by rank, 500 - 4,000 tokens each (tool descriptions count
  as part of the template);
* segment lengths are log-normal with median 300 tokens and sigma 0.8,
  clipped to [16, 8192]; a document of a document-QA request is 4x longer;
* turn 1 prompt = template + user segment; turn t > 1 prompt = the previous
  prompt + the previous response + (agent: a tool-output segment) + a user
  segment; generation = an optional chain-of-thought segment (probability
  0.3) followed by the response; chain-of-thought is not carried into the
  next prompt;
* segment lengths are rounded to whole 16-token blocks, so every block holds
  tokens of one segment and its token-type histogram has one type;
* block hashes chain over the whole sequence from a fixed root,
  h_j = mix64(h_{j-1} xor c_j), c_j a content id of (segment, block index);
  identical content at an identical position gives an identical hash;
* cache hints of a block: shared-prefix for template blocks; multi-turn for a
  request with history or, on turn 1, a predictor output drawn with the
  confusion rates the paper reports for its session predictor (false
  positives 71 of 186, false negatives 15 of 190); conversation for a request
  with history; agentic for agent and tool-use requests; untemplated for
  non-template prompt blocks of a request not flagged multi-turn; decode for
  generated blocks of such a request.
"""
import ctypes
import heapq
import math
import os
import subprocess

import numpy as np

from .pools import M64, MU_AGENT_MS, MU_CHAT_MS, ROOT, SIGMA_AGENT, SIGMA_CHAT, mix64

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "chain.c")
_LIB = os.path.join(_HERE, "libsynth_chain.so")
_chain_fn = None


def build(force=True):
    """Compile chain.c (gcc) into libsynth_chain.so."""
    if not force and os.path.exists(_LIB) and os.path.getmtime(_LIB) >= os.path.getmtime(_SRC):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-std=c99", "-o", tmp, _SRC])
    os.replace(tmp, _LIB)
    return _LIB


def _chain_lib():
    global _chain_fn
    if _chain_fn is None:
        build(force=False)
        L = ctypes.CDLL(_LIB)
        f = L.synth_chain_segment
        f.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p]
        f.restype = ctypes.c_uint64
        _chain_fn = f
    return _chain_fn

SYSTEM, USER, TOOL, RESPONSE, COT = range(5)
# hint byte layout (one byte per block)
H_DECODE, H_UNTEMPLATED, H_MULTI_TURN, H_AGENTIC, H_CONVERSATION, H_SHARED_PREFIX = 1, 2, 4, 8, 16, 32

CATEGORIES = ("chat", "agent", "tool_use", "programming", "doc_qa")
MULTI_TURN = (True, True, False, False, False)
AGENTIC = (False, True, True, False, False)
# Table 2: per-category request shares
MIXES = {
    "multi_turn_dominant": (0.50, 0.30, 0.10, 0.05, 0.05),
    "balanced": (0.30, 0.20, 0.25, 0.15, 0.10),
    "single_turn_dominant": (0.10, 0.10, 0.40, 0.25, 0.15),
}
GAP_S = {0: (4.82, 1.25), 1: (2.28, 1.34)}  # Table 3, chat / agent, ln-seconds

DEFAULTS = dict(
    interval_ms=30, t0=1000, n_templates=2000, zipf_s=1.1, template_tokens=(500, 4000),
    seg_median=300.0, seg_sigma=0.8, seg_clip=(16, 8192), doc_scale=4.0, mean_turns=6.0,
    p_cot=0.3, pred_fp=71.0 / 186.0, pred_fn=15.0 / 190.0, block_tokens=16,
)

GOLD = 0x9E3779B97F4A7C15


def _mix(z):
    z &= M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def chain_segment(h, key, n):
    """Hashes of n blocks of the segment with content key `key`, chained from
    parent hash h: c_j = mix64(key ^ (j+1) G), h_j = mix64(h_{j-1} ^ c_j)."""
    out = np.empty(n, np.uint64)
    last = _chain_lib()(h, key, n, out.ctypes.data)
    return out, int(last)


class _Session:
    __slots__ = ("sid", "cat", "n_turns", "template", "hist_hash", "hist_type", "hist_tmpl", "last_hash", "key")


class TraceGen:
    """One cache instance's request stream; `next()` returns the request of the
    next slot."""

    def __init__(self, mix, seed, **over):
        p = dict(DEFAULTS)
        p.update(over)
        self.p = p
        self.mix = MIXES[mix] if isinstance(mix, str) else tuple(mix)
        self.rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed)))
        self.seed_key = int(mix64(np.uint64(seed & M64) ^ np.uint64(0x5AE5AE5AE5AE5AE5)))
        w = np.asarray(self.mix, np.float64)
        self.cum_cat = np.cumsum(w / w.sum())
        ranks = np.arange(1, p["n_templates"] + 1, dtype=np.float64)
        zw = ranks ** -p["zipf_s"]
        self.cum_template = np.cumsum(zw / zw.sum())
        tr = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 1])))
        lo, hi = p["template_tokens"]
        bt = p["block_tokens"]
        self.template_blocks = np.maximum(1, np.rint(tr.integers(lo, hi + 1, size=p["n_templates"]) / bt)).astype(int)
        self._tcache = {}
        self.slot = 0
        self.due = ([], [])  # due turns of chat / agent sessions
        self.n_sessions = 0

    # ------------------------------------------------------------ pieces
    def _template(self, t):
        """Hashes of template t's blocks (they sit at the root of every prompt)."""
        got = self._tcache.get(t)
        if got is None:
            n = int(self.template_blocks[t])
            key = _mix(self.seed_key ^ (0x7E3A << 32) ^ t)
            got = chain_segment(int(ROOT), key, n)
            self._tcache[t] = got
        return got

    def _seg_blocks(self, scale=1.0):
        p = self.p
        x = p["seg_median"] * scale * math.exp(p["seg_sigma"] * self.rng.standard_normal())
        x = min(max(x, p["seg_clip"][0]), p["seg_clip"][1] * scale)
        return max(1, int(round(x / p["block_tokens"])))

    def _segment(self, sess, turn, idx):
        return _mix(sess.key ^ ((turn << 8) | idx))

    def _draw(self, cum):
        return min(int(np.searchsorted(cum, self.rng.random(), side="right")), len(cum) - 1)

    def _new_session(self, cat):
        s = _Session()
        s.sid = self.n_sessions
        self.n_sessions += 1
        s.cat = cat
        s.n_turns = int(self.rng.geometric(1.0 / self.p["mean_turns"])) if MULTI_TURN[s.cat] else 1
        s.template = self._draw(self.cum_template)
        s.key = _mix(self.seed_key ^ (s.sid + 1) * GOLD)
        s.hist_hash = None
        return s

    # ------------------------------------------------------------ requests
    def next(self):
        p = self.p
        now = p["t0"] + self.slot * p["interval_ms"]
        self.slot += 1
        cat = self._draw(self.cum_cat)
        due = self.due[cat] if MULTI_TURN[cat] else None
        if due and due[0][0] <= now:
            _, _, turn, sess = heapq.heappop(due)
        else:
            sess, turn = self._new_session(cat), 1
        multi = MULTI_TURN[sess.cat]
        if turn == 1:
            th, tlast = self._template(sess.template)
            pre_hash = [th]
            pre_type = [np.full(len(th), SYSTEM, np.uint8)]
            pre_tmpl = [np.ones(len(th), bool)]
            last = tlast
            pred = self.rng.random()
            mt_hint = (pred >= p["pred_fn"]) if multi else (pred < p["pred_fp"])
        else:
            pre_hash, pre_type, pre_tmpl = [sess.hist_hash], [sess.hist_type], [sess.hist_tmpl]
            last = sess.last_hash
            mt_hint = True
        conv = turn > 1
        segs = []
        if turn > 1 and sess.cat == 1:
            segs.append((TOOL, self._seg_blocks()))
        segs.append((USER, self._seg_blocks(p["doc_scale"] if sess.cat == 4 else 1.0)))
        for i, (ty, n) in enumerate(segs):
            h, last = chain_segment(last, self._segment(sess, turn, i), n)
            pre_hash.append(h)
            pre_type.append(np.full(n, ty, np.uint8))
            pre_tmpl.append(np.zeros(n, bool))
        prompt_hash = np.concatenate(pre_hash)
        prompt_type = np.concatenate(pre_type)
        prompt_tmpl = np.concatenate(pre_tmpl)
        prompt_last = last
        gen_hash, gen_type = [], []
        if self.rng.random() < p["p_cot"]:
            n = self._seg_blocks()
            h, last = chain_segment(last, self._segment(sess, turn, 8), n)
            gen_hash.append(h)
            gen_type.append(np.full(n, COT, np.uint8))
        n_resp = self._seg_blocks()
        resp_key = self._segment(sess, turn, 9)
        h, last = chain_segment(last, resp_key, n_resp)
        gen_hash.append(h)
        gen_type.append(np.full(n_resp, RESPONSE, np.uint8))
        gen_hash = np.concatenate(gen_hash)
        gen_type = np.concatenate(gen_type)

        req_bits = (H_MULTI_TURN if mt_hint else 0) | (H_AGENTIC if AGENTIC[sess.cat] else 0) | \
            (H_CONVERSATION if conv else 0)
        single = not (mt_hint or conv)
        hint_p = np.where(prompt_tmpl, H_SHARED_PREFIX, H_UNTEMPLATED if single else 0).astype(np.uint8) | req_bits
        hint_g = np.full(len(gen_hash), (H_DECODE if single else 0) | req_bits, np.uint8)

        if multi and turn < sess.n_turns:
            # next prompt = this prompt + the response (without chain-of-thought)
            rh, rlast = chain_segment(prompt_last, resp_key, n_resp)
            sess.hist_hash = np.concatenate([prompt_hash, rh])
            sess.hist_type = np.concatenate([prompt_type, np.full(n_resp, RESPONSE, np.uint8)])
            sess.hist_tmpl = np.concatenate([prompt_tmpl, np.zeros(n_resp, bool)])
            sess.last_hash = rlast
            mu, sg = GAP_S[sess.cat]
            gap_ms = int(round(1000.0 * math.exp(mu + sg * self.rng.standard_normal())))
            heapq.heappush(self.due[sess.cat], (now + max(gap_ms, 1), sess.sid, turn + 1, sess))
        hashes = np.concatenate([prompt_hash, gen_hash])
        types = np.concatenate([prompt_type, gen_type])
        return dict(now=now, session=sess.sid, turn=turn, category=sess.cat, n_prompt=len(prompt_hash),
                    n_gen=len(gen_hash), hashes=hashes, types=types,
                    hints=np.concatenate([hint_p, hint_g]))


def block_counts(types, block_tokens=16):
    """Token-type histograms [n, 5] of one-type blocks."""
    c = np.zeros((len(types), 5), np.uint8)
    c[np.arange(len(types)), types] = block_tokens
    return c


TRACE_CONFIGS = {
    # 100k requests, balanced mix, one cache of 36K tokens
    "trace_balanced": dict(mix="balanced", n_requests=100_000, n_inst=1, capacity=2250, k_min=1, max_k=1024, K=32,
                           seed=1003, concurrency=4),
    # 256 caches of 65,536 blocks: half single-turn dominant, half multi-turn dominant
    "batched_sweep": dict(mixes=("single_turn_dominant", "multi_turn_dominant"), n_requests=10_000, n_inst=256,
                          capacity=65536, k_min=256, max_k=4096, K=32, seed=1005, concurrency=4),
}


# The paper's four queues of the trace configurations (Sec. 3.1): evict-first,
# structural, chat and agent (kinds 0 evict-first, 1 structural, 2 log-normal),
# their starting timing parameters, and the Classify roles.
TRACE_KINDS = [0, 1, 2, 2]
TRACE_ROLES = [0, 1, 2, 3]
TRACE_MU = [0.0, 0.0, MU_CHAT_MS, MU_AGENT_MS]
TRACE_SIGMA = [1.0, 1.0, SIGMA_CHAT, SIGMA_AGENT]


def trace_gen(name, inst, n_inst=None, **over):
    """Request generator of instance `inst` of trace configuration `name`."""
    cfg = TRACE_CONFIGS[name]
    n_inst = cfg["n_inst"] if n_inst is None else n_inst
    if "mixes" in cfg:
        mix = cfg["mixes"][0 if inst < n_inst // 2 else 1]
    else:
        mix = cfg["mix"]
    return TraceGen(mix, cfg["seed"] * 1000 + inst, **over)


def trace_gens(name, n_inst, **over):
    return [trace_gen(name, i, n_inst, **over) for i in range(n_inst)]

