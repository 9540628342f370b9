"""GPU parity at full size: 4,194,304 blocks, 5 queues, k = 4,096, and 4,096
prefix-match requests of 128 hashes, in the launch configuration the
benchmark times.  Every victim, score bit, decision entry, match length,
counter and pool bit is compared with the oracle, also for the prefix match
and decision issued as one sae_match_select call."""
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


def test_large_select_with_concurrent_prefix_match(large):
    """The large-pool configuration's concurrent case: a read-only prefix match
    of 4,096 requests x 128 hashes on a second stream overlaps the
    score+select pass on the first; both results equal the oracle's."""
    import torch
    p, pool, cfg = large
    R, L = synth.make_requests(pool["chains"], cfg["n_req"], cfg["req_len"], cfg["hit_frac"], 5)
    now = pool["now"] + 1
    hd = torch.as_tensor(np.asarray(R, np.uint64).view(np.int64)).cuda()
    ld = torch.as_tensor(np.asarray(L, np.int32)).cuda()
    ml = torch.full((len(L),), -7, dtype=torch.int32, device="cuda")
    mid = torch.full(hd.shape, -7, dtype=torch.int32, device="cuda")
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    say("large: score_select on stream A, read-only prefix match on stream B")
    p.out.run(p.ctx, now, cfg["k"], 0, stream=sa)
    api.sae_prefix_match(p.ctx, hd, ld, now, 0, ml, matched_ids=mid, stream=sb)
    torch.cuda.synchronize()
    om, omid = p.oc.prefix_match(R, L, now, touch=False, stats=False)
    assert np.array_equal(ml.cpu().numpy(), om), "match lengths differ"
    assert np.array_equal(mid.cpu().numpy(), omid), "matched ids differ"
    lists, key, dec = p.oc.score_select(now, cfg["k"])
    cnt = p.out.count[0].cpu().numpy()
    vic = p.out.victims[0].cpu().numpy()
    sc = p.out.scores[0].cpu().numpy().view(np.uint32)
    for q in range(p.Q):
        c = int(cnt[q])
        assert c == len(lists[q]) and np.array_equal(vic[q, :c], lists[q]), "queue %d differs" % q
        assert np.array_equal(sc[q, :c], key[lists[q]]), "queue %d: score bits differ" % q
    d = int(p.out.decision_count[0])
    assert d == len(dec) and np.array_equal(p.out.decision[0, :d].cpu().numpy(), dec)
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


def test_large_match_select(large):
    """sae_match_select at full size, as the benchmark's step calls it: 4,096
    requests x 128 hashes with touch and statistics, then the committed
    decision of k = 4,096, the selection's sampling and bounds in the prefix
    match's launch; equal to the oracle's prefix match followed by its
    selection, twice in a row."""
    p, pool, cfg = large
    for j, t in enumerate((40, 50)):
        R, L = synth.make_requests(pool["chains"], cfg["n_req"], cfg["req_len"], cfg["hit_frac"], 60 + j)
        say("large: match+select %d" % j)
        om, dec = p.match_select(R, L, pool["now"] + t, api.PM_TOUCH | api.PM_STATS, pool["now"] + t, cfg["k"],
                                 commit=True)
        assert om.sum() > 0 and len(dec) == cfg["k"]
        p.check_counters()
        p.check_pool()
    assert set(p.status()) <= {"SELECT_FALLBACK"}


def test_large_stage_two_decision():
    """Full size with an evict-first queue of about 2,000 blocks, fewer than
    k = 4,096: every decision takes all of that queue's evictable blocks and
    fills the rest from the other queues merged by (P, id) (Algorithm 1's
    second stage, the final kernel's union workgroups), with the pass alone
    and with the combined call, twice in a row with commits."""
    cfg = synth.pool_config("large", mix=[0.0005, 0.35, 0.3, 0.2, 0.1495])
    say("stage two: generating pool")
    pool = synth.make_pool(cfg, seed=4321)
    p = Pair(cfg["kinds"], pool, cfg["k"], mu=cfg["mu"], sigma=cfg["sigma"], K=cfg["k"])
    try:
        say("stage two: score_select")
        _, _, dec = p.select(pool["now"], cfg["k"])
        n_ef = int(np.count_nonzero(pool["queue"] == 0))
        assert n_ef < cfg["k"] and len(dec) == cfg["k"]
        for j, t in enumerate((10, 20)):
            R, L = synth.make_requests(pool["chains"], cfg["n_req"], cfg["req_len"], cfg["hit_frac"], 70 + j)
            say("stage two: match+select %d" % j)
            p.match_select(R, L, pool["now"] + t, api.PM_TOUCH | api.PM_STATS, pool["now"] + t, cfg["k"],
                           commit=True)
            p.check_counters()
            p.check_pool()
        assert set(p.status()) <= {"SELECT_FALLBACK"}
    finally:
        p.close()


def test_large_equal_key_clusters():
    """Blocks added together share last_access, so their keys repeat: here
    last_access takes 400 values, which makes clusters of about 2,000 equal
    keys per (queue, type), and every queue's candidates hold whole clusters.
    Every list and the decision equal the oracle's on the pool-scan engine,
    with no fallback."""
    cfg = synth.pool_config("large")
    pool = synth.make_pool(cfg, seed=1234)
    rng = np.random.default_rng(9)
    la = pool["now"] - 1000 * rng.integers(1, 401, pool["n_blocks"])
    pool["last_access"] = la.astype(pool["last_access"].dtype)
    p = Pair(cfg["kinds"], pool, cfg["k"], mu=cfg["mu"], sigma=cfg["sigma"], K=cfg["k"])
    try:
        for now, k in ((pool["now"], cfg["k"]), (pool["now"] + 500, 1000), (pool["now"] + 900, 4000)):
            say("large clusters: score_select k=%d" % k)
            p.select(now, k, api.SS_ENGINE_SCAN)
            assert not p.status()
    finally:
        p.close()
