"""GPU parity on trace replay, with the oracle replaying beside the GPU.

* Balanced mix (Table 2), one cache of 2,250 blocks (36K tokens): every step's
  match length and every eviction decision equal the oracle's; counters,
  learned weights and the whole pool state (valid, leaf and reference bits,
  child counts, access times) agree.  Learner sets and decision modes that
  the full-length runs (tests/test_gpu_trace_full.py) do not cover: fixed
  weights, the appendix text's rules, cascading decisions.
* Batched sweep: 256 caches of 65,536 blocks in one context, decisions of at
  least 256 victims, two instances (one of each half) replayed by the oracle:
  every learner with interval recording across 256 instances, and cascading
  decisions."""
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
