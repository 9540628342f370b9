"""GPU parity on the full-length trace replays, against digests the oracle wrote.

* Balanced mix (Table 2), 100,000 requests on one 36K-token cache, once with
  Algorithms 2 and 3 and once with Algorithms 2, 3, 4 and the decay-power
  learner.
* Batched sweep, 10,000 requests on each of 256 caches of 65,536 blocks in
  one context (128 single-turn-dominant, 128 multi-turn-dominant traces), once
  with fixed weights and once with Algorithms 2 and 3; eight caches (four of
  each half) are compared.

tests/golden/make_trace_digests.py replayed the compared caches on the oracle
and stored, per step, a chained digest of the match length and every eviction
decision (tests/trace_digest.py), and every 1,000 steps the counters and the
bits of the learned parameters.  The HIP replay computes the same digests; the
first step whose digest differs is named, and every checkpoint must be equal.
The four replays run side by side, each in a process of its own
(tests/trace_full_run.py), since the host side of a replay step is what takes
the time: about 8 minutes in all on one MI355X (each balanced replay makes
about 7.6 million eviction decisions, one host round trip each).
"""
import json
import os
import subprocess
import sys
import threading
import time

import pytest

pytestmark = pytest.mark.gpu

from harness import say  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))
RUNS = ["balanced_alg23", "balanced_all", "sweep_fixed", "sweep_learned"]
LIMIT_S = 900


def test_full_length_replays():
    procs, results, lines = {}, {}, []
    lock = threading.Lock()

    def pump(name, p):
        for ln in p.stdout:
            ln = ln.rstrip("\n")
            with lock:
                lines.append((name, ln))
            if ln.startswith("RESULT "):
                results[name] = json.loads(ln[7:])
            else:
                say("[%s] %s" % (name, ln))

    threads = []
    for n in RUNS:
        p = subprocess.Popen([sys.executable, "-u", os.path.join(HERE, "trace_full_run.py"), n],
                             stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
        procs[n] = p
        t = threading.Thread(target=pump, args=(n, p), daemon=True)
        t.start()
        threads.append(t)
    t0 = time.time()
    try:
        for n, p in procs.items():
            p.wait(timeout=max(1.0, LIMIT_S - (time.time() - t0)))
    finally:
        for p in procs.values():
            if p.poll() is None:
                p.kill()
                p.wait()
    for t in threads:
        t.join(timeout=10)
    bad = {n: p.returncode for n, p in procs.items() if p.returncode != 0}
    assert not bad, "replays failed: %s\n%s" % (bad, "\n".join("[%s] %s" % x for x in lines[-40:]))
    assert set(results) == set(RUNS)
    for n in RUNS:
        say("%s: %.0f s, %s" % (n, results[n]["seconds"], results[n]["all"]))
    fixed, learned = results["sweep_fixed"]["halves"], results["sweep_learned"]["halves"]
    for h in fixed:
        f, l = fixed[h], learned[h]
        say("%s: block hit ratio fixed %.4f, learned %.4f; prefill tokens fixed %d, learned %d"
            % (h, f["block_hit_ratio"], l["block_hit_ratio"], f["prefill_tokens"], l["prefill_tokens"]))
