"""Step digests of a trace replay, for full-length parity against stored files.

A replay step of one cache instance yields its prefix-match length and the
eviction decisions it took (block ids, in decision order).  The digest of a
run is a chain over the steps: state_s = blake2b-64(state_{s-1} || record_s),
record_s = (step, match length, number of decisions, each decision's length
and ids) as little-endian int32.  Per step the low 16 bits of the state are
stored; because the state chains, the first stored value that differs names
the step where two runs first differ.  Every CHECK_EVERY steps (and after the
last) a checkpoint holds the full state, the instance's feedback counters and
the bits of its learned parameters.

The run definitions below are shared by the generator that writes the stored
files from the oracle (tests/golden/make_trace_digests.py) and by the GPU test
that replays the same runs on the HIP path.  This module holds no step of the
eviction method.
"""
import hashlib
import json
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
DIGEST_DIR = os.path.join(HERE, "golden", "trace_digests")
CHECK_EVERY = 1000

# name -> (trace configuration, steps, learner bits, instances compared)
#  learner bits: 1 Algorithm 3, 2 Algorithm 2, 4 Algorithm 4, 8 decay power
RUNS = {
    # the balanced-mix trace replay, 100k requests on one 36K-token cache
    "balanced_alg23": dict(trace="trace_balanced", steps=100_000, learn=3, insts=[0]),
    "balanced_all": dict(trace="trace_balanced", steps=100_000, learn=15, insts=[0]),
    # the batched sweep, 10k requests on each of 256 caches of 65,536 blocks;
    # instances 0-127 run single-turn-dominant traces, 128-255 multi-turn-dominant
    "sweep_learned": dict(trace="batched_sweep", steps=10_000, learn=3, insts=[0, 41, 86, 127, 128, 169, 214, 255]),
    "sweep_fixed": dict(trace="batched_sweep", steps=10_000, learn=0, insts=[0, 41, 86, 127, 128, 169, 214, 255]),
}

COUNTER_KEYS = ("evicted", "missed", "hits", "evictions", "ev_count", "pending", "n_updates", "bin_hits",
                "bin_missed", "type_hits", "type_added", "resident")


class Chain:
    """The chained digest of one instance's replay."""

    def __init__(self, steps):
        self.state = b"\0" * 8
        self.low = np.zeros(steps, np.uint16)

    def add(self, step, match_len, decisions):
        parts = [np.array([step, match_len, len(decisions)], "<i4").tobytes()]
        for d in decisions:
            d = np.asarray(d, "<i4")
            parts.append(np.array([len(d)], "<i4").tobytes())
            parts.append(d.tobytes())
        self.state = hashlib.blake2b(self.state + b"".join(parts), digest_size=8).digest()
        self.low[step] = int.from_bytes(self.state[:2], "little")

    def hex(self):
        return self.state.hex()


def f32_bits(a):
    return [int(x) for x in np.asarray(a, np.float32).view(np.uint32).ravel()]


def checkpoint(step, chain, backend, inst, summary):
    """What is compared every CHECK_EVERY steps: digest state, counters,
    learned-parameter bits and the replay's running totals."""
    c = backend.counters(inst)
    w, a = backend.params(inst)
    mu, sg, gm = backend.timing_params(inst)
    cnt = {k: (list(map(int, c[k])) if isinstance(c[k], (list, tuple, np.ndarray)) else int(c[k]))
           for k in COUNTER_KEYS}
    return dict(step=int(step), state=chain.hex(), counters=cnt, w=f32_bits(w), alpha=f32_bits(a), mu=f32_bits(mu),
                sigma=f32_bits(sg), gamma=f32_bits([gm])[0], summary=summary)


def paths(name):
    return os.path.join(DIGEST_DIR, name + ".npz"), os.path.join(DIGEST_DIR, name + ".json")


def save(name, meta, lows, checks):
    """lows: {inst: uint16[steps]}; checks: {inst: [checkpoint, ...]}."""
    os.makedirs(DIGEST_DIR, exist_ok=True)
    npz, js = paths(name)
    np.savez_compressed(npz, **{"inst%d" % i: v for i, v in lows.items()})
    with open(js, "w") as f:
        json.dump(dict(meta, checkpoints={str(i): v for i, v in checks.items()}), f, indent=0, sort_keys=True)
        f.write("\n")


def load(name):
    npz, js = paths(name)
    with np.load(npz) as z:
        lows = {int(k[4:]): z[k].copy() for k in z.files}
    with open(js) as f:
        meta = json.load(f)
    checks = {int(i): v for i, v in meta.pop("checkpoints").items()}
    return meta, lows, checks


def first_difference(a, b):
    """First key where two checkpoints differ (None if equal)."""
    for k in ("state", "counters", "w", "alpha", "mu", "sigma", "gamma", "summary"):
        if a.get(k) != b.get(k):
            return k
    return None
