"""One full-length trace replay on the HIP path, checked against the stored
oracle digests (tests/trace_digest.py RUNS).  Run as a child process by
tests/test_gpu_trace_full.py:

    python tests/trace_full_run.py RUN

Prints a progress line every `report` steps and, at the end, one line
"RESULT <json>" with the replay's totals (per half of a batched sweep).  Exits
non-zero at the first step whose digest differs from the oracle's (naming it),
or at a checkpoint whose counters or learned-parameter bits differ.
"""
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
for p in (ROOT, HERE):
    if p not in sys.path:
        sys.path.insert(0, p)

import trace_digest as td  # noqa: E402
from synth.replay import Replay  # noqa: E402
from synth.trace import TRACE_CONFIGS  # noqa: E402
from trace_setup import KINDS, MU, ROLES, SIGMA, trace_gens  # noqa: E402

STAT_KEYS = ("requests", "prompt_blocks", "hit_blocks", "inserted", "evicted", "decisions", "not_cached")


def say(*a):
    print(*a, flush=True)


def replay(name):
    from paper_2605_18825_amd.engine import DeviceBackend
    run = td.RUNS[name]
    cfg = TRACE_CONFIGS[run["trace"]]
    steps, n_inst = run["steps"], cfg["n_inst"]
    meta, lows, checks = td.load(name)
    assert meta["steps"] == steps and meta["learn"] == run["learn"] and meta["insts"] == run["insts"], meta
    checks = {i: {c["step"]: c for c in v} for i, v in checks.items()}
    report = max(1, steps // 10)
    gens = trace_gens(run["trace"], n_inst)
    dev = DeviceBackend(n_inst, cfg["capacity"], KINDS, ROLES, cfg["max_k"], MU, SIGMA, cfg["K"], run["learn"])
    try:
        rep = Replay(dev, n_inst, cfg["capacity"], cfg["k_min"], cfg["max_k"], cfg["concurrency"])
        chains = {i: td.Chain(steps) for i in run["insts"]}
        t0 = time.time()
        for s in range(steps):
            out = rep.step({i: g.next() for i, g in enumerate(gens)})
            for i in run["insts"]:
                ml, dec = out[i]
                ch = chains[i]
                ch.add(s, ml, dec)
                if ch.low[s] != lows[i][s]:
                    raise AssertionError("%s: instance %d first differs from the oracle at step %d (match length "
                                         "%d, %d decisions)" % (name, i, s, ml, len(dec)))
                if s in checks[i]:
                    sm = rep.summary([i])
                    got = td.checkpoint(s, ch, dev, i, {k: int(sm[k]) for k in STAT_KEYS})
                    k = td.first_difference(got, checks[i][s])
                    if k is not None:
                        raise AssertionError("%s: instance %d at step %d: %s %s vs oracle %s"
                                             % (name, i, s, k, got.get(k), checks[i][s].get(k)))
            if (s + 1) % report == 0:
                say("%s: %d of %d steps equal (%.0f s)" % (name, s + 1, steps, time.time() - t0))
        st = dev.status()
        assert set(st) <= {"SELECT_FALLBACK"}, (name, st)
        res = dict(run=name, seconds=time.time() - t0, all=rep.summary())
        if "mixes" in cfg:
            half = n_inst // 2
            res["halves"] = {cfg["mixes"][0]: rep.summary(list(range(half))),
                             cfg["mixes"][1]: rep.summary(list(range(half, n_inst)))}
        say("RESULT " + json.dumps(res))
    finally:
        dev.close()


if __name__ == "__main__":
    replay(sys.argv[1])
