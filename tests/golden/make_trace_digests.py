"""Write the stored step digests of the full-length trace replays (oracle only).

    python tests/golden/make_trace_digests.py [run ...] [--jobs N]

For every run of tests/trace_digest.py RUNS (all when none is named) the
oracle replays each compared instance for the run's full length: the balanced
trace's 100,000 requests on one cache, and the batched sweep's 10,000
requests on each of its compared caches (every cache of the sweep is
independent of the others, so each is replayed on its own).  The per-step
digests and the checkpoints go to tests/golden/trace_digests/<run>.{npz,json}.

Imports the oracle, the seeded generators and the replay driver only; nothing
from the HIP package.  CPU time: about 17 minutes per balanced run and 3 per
sweep instance on one core; runs and instances are spread over --jobs
processes.
"""
import argparse
import multiprocessing as mp
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
TESTS = os.path.dirname(HERE)
ROOT = os.path.dirname(TESTS)
for p in (ROOT, TESTS):
    if p not in sys.path:
        sys.path.insert(0, p)

import trace_digest as td  # noqa: E402
from oracle_backend import OracleBackend  # noqa: E402
from synth.replay import Replay  # noqa: E402
from synth.trace import TRACE_CONFIGS  # noqa: E402
from trace_setup import KINDS, MU, ROLES, SIGMA, trace_gen  # noqa: E402

STAT_KEYS = ("requests", "prompt_blocks", "hit_blocks", "inserted", "evicted", "decisions", "not_cached")


def summary_of(replay, inst):
    s = replay.summary([inst])
    return {k: int(s[k]) for k in STAT_KEYS}


def replay_instance(job):
    name, inst = job
    run = td.RUNS[name]
    cfg = TRACE_CONFIGS[run["trace"]]
    steps = run["steps"]
    gen = trace_gen(run["trace"], inst)
    orc = OracleBackend([inst], cfg["capacity"], KINDS, ROLES, MU, SIGMA, cfg["K"], run["learn"])
    rep = Replay(orc, cfg["n_inst"], cfg["capacity"], cfg["k_min"], cfg["max_k"], cfg["concurrency"], insts=[inst])
    chain = td.Chain(steps)
    checks = []
    t0 = time.time()
    for s in range(steps):
        r = gen.next()
        ml, dec = rep.step({inst: r})[inst]
        chain.add(s, ml, dec)
        if (s + 1) % td.CHECK_EVERY == 0 or s == steps - 1:
            checks.append(td.checkpoint(s, chain, orc, inst, summary_of(rep, inst)))
        if (s + 1) % 10_000 == 0:
            print("%s instance %d: %d steps, %.0f s" % (name, inst, s + 1, time.time() - t0), flush=True)
    return name, inst, chain.low, checks


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("runs", nargs="*", default=sorted(td.RUNS))
    ap.add_argument("--jobs", type=int, default=max(1, (os.cpu_count() or 2) - 1))
    args = ap.parse_args()
    jobs = [(n, i) for n in args.runs for i in td.RUNS[n]["insts"]]
    # the longest jobs (one cache, 100k requests) first
    jobs.sort(key=lambda j: -td.RUNS[j[0]]["steps"])
    lows = {n: {} for n in args.runs}
    checks = {n: {} for n in args.runs}
    with mp.Pool(min(args.jobs, len(jobs))) as pool:
        for name, inst, low, ch in pool.imap_unordered(replay_instance, jobs):
            lows[name][inst] = low
            checks[name][inst] = ch
            if len(lows[name]) == len(td.RUNS[name]["insts"]):
                run = td.RUNS[name]
                meta = dict(run=name, trace=run["trace"], steps=run["steps"], learn=run["learn"],
                            insts=run["insts"], check_every=td.CHECK_EVERY,
                            written_by="tests/golden/make_trace_digests.py (oracle replay)")
                td.save(name, meta, lows[name], checks[name])
                print("wrote", name, flush=True)


if __name__ == "__main__":
    main()
