"""GPU parity of the pool scan's exact pruning filter at a real k, under the
parameters and block features where its proof has edge cases.  The scan
engine is forced, every victim and score bit is compared with the oracle, and
the exact slow path must not have run: a filter that dropped a candidate
would either change a victim list or starve a queue into that slow path."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

import synth  # noqa: E402
from harness import Pair, say  # noqa: E402
from paper_2605_18825_amd import api  # noqa: E402

LN, STRUCT, REC, EF = 2, 1, 3, 0
N = 65536


def pool_of(kinds, mix, seed):
    cfg = synth.pool_config("tiny", kinds=kinds, mix=mix)
    return synth.make_pool(cfg, n_blocks=N, seed=seed)


def stats(pair):
    return [dict(zip(("evictable", "candidates", "beyond_stripes", "slow"), s)) for s in api.sae_select_stats(pair.ctx, 0, pair.Q)]


def run(pair, pool, k, rounds=3, commit=False, expect_fallback=False):
    try:
        for i in range(rounds):
            pair.select(pool["now"] + 1000 * i, k, api.SS_ENGINE_SCAN, commit=commit)
            st = pair.status()
            if not expect_fallback:
                assert "SELECT_FALLBACK" not in st, "the exact slow path ran (round %d): %s" % (i, stats(pair))
    finally:
        pair.close()


def test_small_sigma_zero_scores():
    """sigma = 0.3: every block beyond dt ~ 1.3e5 has P = 0 exactly (erfc = 0),
    so the bound is (0, id) and the log-normal threshold uses its 2^-100 floor."""
    pool = pool_of([LN, STRUCT, REC], [0.6, 0.2, 0.2], 7001)
    say("pruning: small sigma")
    run(Pair([LN, STRUCT, REC], pool, 512, mu=[8.0, 0, 0], sigma=[0.3, 1, 1]), pool, 512)


def test_extreme_weights():
    """Token and queue weights far outside [2^-90, 2^100] for some (queue,
    type) pairs: the product test is switched off there, the rest prunes."""
    pool = pool_of([LN, STRUCT, REC], [0.3, 0.4, 0.3], 7002)
    w = [1e-30, 1e-3, 1.0, 40.0, 4.99]
    say("pruning: extreme weights")
    run(Pair([LN, STRUCT, REC], pool, 512, mu=[11.7, 0, 0], sigma=[1.25, 1, 1], w=w, alpha=[1e-9, 3.0, 2.5]),
        pool, 512)


def test_gamma_not_one():
    """gamma != 1: structural blocks are never pruned by the product test."""
    pool = pool_of([STRUCT, REC], [0.7, 0.3], 7003)
    say("pruning: gamma 0.5")
    run(Pair([STRUCT, REC], pool, 512, gamma=0.5), pool, 512)


def test_structural_edge_offsets():
    """o_max = 0 (p = 1), last blocks o_b = o_max (p = 0, P = 0), and o_b = 0."""
    pool = pool_of([STRUCT, REC], [0.8, 0.2], 7004)
    rng = np.random.default_rng(4)
    sel = rng.random(N)
    pool["omax"][sel < 0.2] = 0
    pool["ob"][sel < 0.2] = 0
    last = (sel >= 0.2) & (sel < 0.25)
    pool["ob"][last] = pool["omax"][last]
    first = (sel >= 0.25) & (sel < 0.35)
    pool["ob"][first] = 0
    say("pruning: structural offsets")
    run(Pair([STRUCT, REC], pool, 512), pool, 512)


def test_recent_future_and_tied_blocks():
    """dt = 0 (P = +inf), blocks accessed after `now` (scored as dt = 0, status
    bit), and many blocks sharing one last_access (ties by id)."""
    pool = pool_of([LN, STRUCT, REC], [0.4, 0.3, 0.3], 7005)
    rng = np.random.default_rng(5)
    sel = rng.random(N)
    now = pool["now"]
    pool["last_access"][sel < 0.05] = now
    pool["last_access"][(sel >= 0.05) & (sel < 0.08)] = now + 77
    tie = (sel >= 0.08) & (sel < 0.5)
    pool["last_access"][tie] = 12345
    say("pruning: recent, future and tied blocks")
    p = Pair([LN, STRUCT, REC], pool, 512, mu=[11.7, 0, 0], sigma=[1.25, 1, 1])
    try:
        p.select(now, 512, api.SS_ENGINE_SCAN)
        st = p.status()
        assert "SELECT_FALLBACK" not in st, stats(p)
        assert "FUTURE_ACCESS" in st, st
    finally:
        p.close()


def test_evict_first_num_tokens():
    """Evict-first keys are num_tokens (1..16, ties by id): the scan's id
    limit per num_tokens value."""
    pool = pool_of([EF, LN, REC], [0.5, 0.3, 0.2], 7006)
    rng = np.random.default_rng(6)
    pool["ntok"] = rng.integers(1, 17, N).astype(np.int32)
    say("pruning: evict-first num_tokens")
    run(Pair([EF, LN, REC], pool, 512, mu=[0, 9.19, 0], sigma=[1, 1.34, 1]), pool, 512)


def test_small_queue_takes_all():
    """A queue with fewer evictable blocks than k: its bound admits all."""
    pool = pool_of([LN, STRUCT, REC], [0.49, 0.49, 0.02], 7007)
    say("pruning: small queue")
    run(Pair([LN, STRUCT, REC], pool, 512, mu=[11.7, 0, 0], sigma=[1.25, 1, 1]), pool, 512)


def test_large_k():
    """k = 2048 against a 16,384-block sample of a 65,536-block pool: the
    bound sits at sample rank ~700 and its candidates fill many buckets."""
    pool = pool_of([LN, STRUCT, REC], [0.49, 0.49, 0.02], 7007)
    say("pruning: large k")
    run(Pair([LN, STRUCT, REC], pool, 2048, mu=[11.7, 0, 0], sigma=[1.25, 1, 1]), pool, 2048, rounds=1)


def test_learned_weights_between_decisions():
    """Decisions with commit and feedback: the learners move w and alpha, and
    the filter tables follow."""
    pool = pool_of([LN, STRUCT, REC], [0.5, 0.3, 0.2], 7008)
    say("pruning: decisions with learning")
    p = Pair([LN, STRUCT, REC], pool, 512, mu=[11.7, 0, 0], sigma=[1.25, 1, 1], K=512)
    try:
        now = pool["now"]
        for i in range(4):
            p.select(now, 512, api.SS_ENGINE_SCAN, commit=True)
            assert "SELECT_FALLBACK" not in p.status(), stats(p)
            p.feedback(force=True)
            p.check_params()
            now += 1000
    finally:
        p.close()
