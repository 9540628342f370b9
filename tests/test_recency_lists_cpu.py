"""The recency-list selection (oracle/recency.py, the per-queue heap idea of
Sec. 3.2 / Algorithm 1) against the oracle's full sort: identical per-queue
lists, keys and decisions on random pools with ties in last_access, blocks
with dt = 0 (P = +inf), log-normal tails where P is 0 or subnormal, k from 0 to
the whole pool, with the default prefill and with tiny ones (where the walk's
stopping rule decides); and it scores only a small part of the log-normal and
recency queues when k is small."""
import numpy as np
import pytest

import oracle
from oracle.recency import RecencyLists

KINDS = [oracle.EVICT_FIRST, oracle.STRUCTURAL, oracle.LOGNORMAL, oracle.LOGNORMAL, oracle.RECENCY]
NOW = 1_000_000


def make_cache(seed, N, mu, sigma, la_levels=None, w=None, alpha=None, gamma=1.0):
    rng = np.random.default_rng(seed)
    Q = len(KINDS)
    w = rng.uniform(0.1, 5.0, 5) if w is None else w
    alpha = rng.uniform(0.1, 3.0, Q) if alpha is None else alpha
    prm = oracle.Params(Q, w=w, alpha=alpha, mu=mu, sigma=sigma, gamma=gamma, K=0)
    c = oracle.OracleCache(N, KINDS, prm)
    if la_levels is None:
        la = rng.integers(0, NOW, N)
    else:  # few distinct values: many ties
        la = rng.choice(la_levels, N)
    la[rng.random(N) < 0.01] = NOW          # dt = 0: P = +inf
    la[rng.random(N) < 0.005] = NOW + 5     # last_access after now: dt clamps to 0
    queue = rng.choice(Q, N, p=[0.1, 0.3, 0.3, 0.2, 0.1])
    tau = rng.integers(0, 5, N)
    ntok = rng.integers(1, 17, N)
    omax = rng.integers(0, 251, N)
    ob = (rng.random(N) * (omax + 1)).astype(np.int64)
    valid = rng.random(N) < 0.97
    ref = (rng.random(N) < 0.1).astype(np.int32)
    parent = np.full(N, -1, np.int32)
    nl = rng.random(N) < 0.2  # some blocks parent a random other block: not leaves
    parent[nl] = rng.integers(0, N, int(nl.sum()))
    parent[parent == np.arange(N)] = -1
    h = rng.integers(1, 2**63, N, dtype=np.int64).astype(np.uint64)
    c.bind(la.astype(np.int32), queue.astype(np.int32), tau.astype(np.int32), ntok.astype(np.int32),
           ob.astype(np.int32), omax.astype(np.int32), valid, ref, parent, h, None)
    return c


def check_equal(c, k, prefills=(None, 1, 0)):
    """The default prefill (k per list), and prefills so small that the walk's
    stopping rule decides almost every block."""
    lists, key, dec = c.score_select(NOW, k)
    rl = RecencyLists(c)
    for pf in prefills:
        rlists, rkeys, rdec = rl.score_select(NOW, k, prefill=pf)
        for q in range(c.Q):
            assert np.array_equal(rlists[q], lists[q]), "queue %d differs (k=%d, prefill %s)" % (q, k, pf)
            assert np.array_equal(rkeys[q], key[lists[q]]), "queue %d keys differ" % q
        assert np.array_equal(rdec, dec)
    rl.score_select(NOW, k)
    return rl


@pytest.mark.parametrize("seed", [1, 2, 3])
@pytest.mark.parametrize("k", [0, 1, 10, 257, 4096])
def test_matches_full_sort(seed, k):
    c = make_cache(seed, 30_000, mu=[0, 0, 11.727755, 9.187755, 0], sigma=[1, 1, 1.25, 1.34, 1])
    check_equal(c, k)


@pytest.mark.parametrize("k", [64, 3000, 40_000])
def test_ties_in_last_access(k):
    levels = np.arange(0, NOW, 50_000)  # 20 distinct times
    c = make_cache(7, 40_000, mu=[0, 0, 11.7, 9.2, 0], sigma=[1, 1, 1.25, 1.34, 1], la_levels=levels)
    check_equal(c, k)


@pytest.mark.parametrize("k", [16, 500, 5000])
def test_zero_and_subnormal_tails(k):
    # sigma 0.5 around mu = 5: u = (ln dt - 5) / 0.7071 passes 9 (p = 0, P = 0) near
    # dt = e^11.4 ~ 90,000 and leaves a band of subnormal P just below it
    c = make_cache(11, 30_000, mu=[0, 0, 5.0, 5.0, 0], sigma=[1, 1, 0.5, 0.5, 1],
                   w=np.full(5, 0.1, np.float32), alpha=np.full(5, 0.1, np.float32))
    key, _ = c.keys(NOW)
    P = key.view(np.float32)
    ln = np.isin(c.queue, [2, 3]) & c.evictable()
    assert (P[ln] == 0).sum() > 1000, "the pool holds P = 0 ties"
    sub = ln & (P > 0) & (P < np.float32(2.0 ** -126))
    assert sub.sum() > 0, "the pool holds subnormal P"
    check_equal(c, k)


def test_walk_visits_few_blocks():
    c = make_cache(5, 200_000, mu=[0, 0, 11.727755, 9.187755, 0], sigma=[1, 1, 1.25, 1.34, 1])
    rl = check_equal(c, 64)
    ev = c.evictable()
    lnrec = int((ev & np.isin(c.queue, [2, 3, 4])).sum())
    struct = int((ev & (c.queue == 1)).sum())
    walked = rl.visited - struct  # the structural queue is scanned whole
    assert walked < 0.05 * lnrec, (walked, lnrec)


def test_nothing_evictable_and_one_queue():
    """Every block referenced: every list empty, the decision empty; then
    only one log-normal queue holds evictable blocks."""
    c = make_cache(13, 5_000, mu=[0, 0, 11.7, 9.2, 0], sigma=[1, 1, 1.25, 1.34, 1])
    c.ref_count[:] = 1
    rl = check_equal(c, 64)
    assert rl.visited == 0
    _, _, dec = rl.score_select(NOW, 64)
    assert dec.size == 0
    c.ref_count[:] = np.where(c.queue == 2, 0, 1)
    check_equal(c, 64)
    check_equal(c, 100_000)
