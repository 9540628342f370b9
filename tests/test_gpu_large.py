"""GPU parity at full size: 4,194,304 blocks, 5 queues, k = 4,096, and 4,096
prefix-match requests of 128 hashes, in the launch configuration the
benchmark times.  Every victim, score bit, decision entry, match length,
counter and pool bit is compared with the oracle."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

import synth  # noqa: E402
from harness import Pair, say  # noqa: E402
from paper_2605_18825_amd import api  # noqa: E402


@pytest.fixture(scope="module")
def large():
    cfg = synth.pool_config("large")
    say("large: generating pool")
    pool = synth.make_pool(cfg)
    p = Pair(cfg["kinds"], pool, cfg["k"], mu=cfg["mu"], sigma=cfg["sigma"], K=cfg["k"])
    yield p, pool, cfg
    p.close()


def test_large_select_no_commit(large):
    p, pool, cfg = large
    say("large: score_select k=4096")
    p.select(pool["now"], cfg["k"])
    assert not p.status()


def test_large_fallback_path(large):
    p, pool, cfg = large
    say("large: exact slow path")
    p.select(pool["now"] + 3, cfg["k"], api.SS_FORCE_FALLBACK)
    assert p.status() == ["SELECT_FALLBACK"]


def test_large_match_commit_feedback(large):
    p, pool, cfg = large
    R, L = synth.make_requests(pool["chains"], cfg["n_req"], cfg["req_len"], cfg["hit_frac"], 4)
    say("large: prefix match 4096 x 128")
    m = p.prefix_match(R, L, pool["now"] + 10, api.PM_TOUCH | api.PM_STATS)
    assert m.sum() > 0
    say("large: decision + commit")
    p.select(pool["now"] + 20, cfg["k"], commit=True)
    p.check_counters()
    p.check_pool()
    p.feedback()
    p.check_params()
    say("large: second decision")
    p.select(pool["now"] + 30, cfg["k"], commit=True)
    p.check_counters()
