"""GPU parity on trace replay.

* Balanced mix (Table 2), one cache of 2,250 blocks (36K tokens), online
  learning on: every step's match length and every eviction decision equal the
  oracle's; counters, learned weights and the pool state agree.
* Batched sweep: 256 caches of 65,536 blocks in one context (half
  single-turn-dominated, half multi-turn-dominated traces), decisions of at
  least 256 victims; two sampled instances (one of each half) are replayed by
  the oracle beside the GPU and compared the same way."""
import pytest

pytestmark = pytest.mark.gpu

from trace_pair import run_pair  # noqa: E402


def test_trace_balanced_first_1500_requests():
    rd, ro, _ = run_pair("trace_balanced", 1500, [0], check_every=250)
    s = rd.summary()
    assert s["evicted"] > 0 and s["hit_blocks"] > 0


def test_trace_balanced_fixed_weights():
    rd, ro, _ = run_pair("trace_balanced", 400, [0], learn=0, check_every=200)
    assert rd.summary()["evicted"] > 0


def test_trace_balanced_all_learners():
    """Algorithms 2, 3 and 4 and the decay-power learner together: every
    step's matches and decisions, and mu / sigma / gamma, agree bit for bit."""
    rd, ro, _ = run_pair("trace_balanced", 1200, [0], learn=15, check_every=200)
    o = ro.be.c[0]
    assert o.n_updates > 0 and len(o.ivl[2]) + len(o.ivl[3]) > 0


def test_trace_balanced_text_rules():
    """The appendix text's token and queue rules with Algorithm 4 and the
    decay power, from the paper's initial token weights."""
    rd, ro, _ = run_pair("trace_balanced", 1200, [0], learn=60, check_every=200, w=[2.0, 1.5, 1.0, 1.0, 0.1])
    assert ro.be.c[0].n_updates > 0


def test_trace_balanced_cascading_decisions():
    """Algorithm 1 one victim at a time (SAE_SS_CASCADE) on the balanced
    trace: every decision equals the oracle's sequential cascade."""
    rd, ro, _ = run_pair("trace_balanced", 1500, [0], check_every=250, cascade=True)
    assert rd.summary()["evicted"] > 0


def test_batched_sweep_cascading_decisions():
    rd, ro, _ = run_pair("batched_sweep", 900, [5, 200], check_every=300, cascade=True)
    assert rd.summary()["evicted"] > 0


def test_batched_sweep_all_learners():
    """Interval placement across 256 instances of one context."""
    rd, ro, _ = run_pair("batched_sweep", 900, [5, 200], learn=15, check_every=300)
    assert rd.summary()["evicted"] > 0
    assert all(len(ro.be.c[i].ivl[2]) + len(ro.be.c[i].ivl[3]) > 0 for i in (5, 200))


def test_batched_sweep_sampled_instances():
    rd, ro, _ = run_pair("batched_sweep", 900, [5, 200], check_every=150)
    s = rd.summary()
    assert s["evicted"] > 0 and s["decisions"] > 0
