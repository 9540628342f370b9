"""Sequential cascading eviction (Algorithm 1's Evict() one victim at a time,
with a parent that loses its last child evictable for the next call) against
the snapshot decision the HIP path takes: the oracle's two cascade versions
agree, the cascade reduces to the snapshot decision when no parent can be
promoted, and what batching changes is measured on the synthetic pool and on
trace replay (printed)."""
import numpy as np
import pytest

import synth
from oracle import OracleCache, Params
from oracle.policy import EVICT_FIRST, LOGNORMAL, RECENCY, STRUCTURAL
from oracle_backend import OracleBackend
from synth.replay import Replay
from synth.trace import TraceGen

KINDS = [EVICT_FIRST, STRUCTURAL, LOGNORMAL, RECENCY]


@pytest.fixture(scope="module", autouse=True)
def _built(oracle_lib):
    return oracle_lib


def chain_cache(seed, n=48, L=3, ef=True):
    rng = np.random.default_rng(seed)
    kinds = KINDS if ef else KINDS[1:]
    c = OracleCache(n, kinds, Params(len(kinds), mu=[0, 0, 9.0, 0][-len(kinds):], sigma=1.2, K=1000))
    parent = np.array([-1 if b % L == 0 else b - 1 for b in range(n)], np.int32)   # roots first in a chain
    hashes = rng.integers(1, 2 ** 62, n, dtype=np.uint64)
    la = rng.integers(0, 5000, n)
    la[rng.random(n) < 0.2] = 777                                                # ties
    c.bind(la, rng.integers(0, len(kinds), n), rng.integers(0, 5, n), rng.integers(1, 17, n),
           rng.integers(0, 20, n), np.full(n, 20), rng.random(n) < 0.95, (rng.random(n) < 0.1).astype(np.int32),
           parent, hashes)
    return c


@pytest.mark.parametrize("seed", range(8))
def test_cascade_heap_equals_literal(seed):
    c = chain_cache(seed, ef=seed % 2 == 0)
    for k in (1, 5, 17, 48):
        a = c.cascade_literal(6000, k)
        b = c.decide_cascade(6000, k)
        assert np.array_equal(a, b), (k, a, b)


def test_cascade_reduces_to_snapshot_without_parents():
    c = chain_cache(3, L=1)
    for k in (1, 7, 30):
        lists, key, dec = c.score_select(6000, k)
        assert np.array_equal(c.decide_cascade(6000, k), dec)


def test_cascade_promotes_within_a_decision():
    """Chain root 0 <- 1 <- 2 (leaf): the root and its child are far older than
    the other leaves, so the cascade takes 2, then 1, then 0; the snapshot
    decision can only take the leaf 2 and then other leaves."""
    c = OracleCache(6, [RECENCY], Params(1))
    c.bind([10, 5, 900, 950, 960, 970], [0] * 6, [0] * 6, [16] * 6, [0] * 6, [0] * 6, [True] * 6, [0] * 6,
           [-1, 0, 1, -1, -1, -1], np.arange(1, 7, dtype=np.uint64))
    assert c.decide_cascade(1000, 3).tolist() == [2, 1, 0]
    assert c.score_select(1000, 3)[2].tolist() == [2, 3, 4]
    c.commit(c.decide_cascade(1000, 3))
    assert not c.valid[:3].any() and c.valid[3:].all()


def test_what_batching_changes_on_the_synthetic_pool():
    cfg = synth.pool_config("tiny")
    pool = synth.make_pool(cfg)
    c = OracleCache(pool["n_blocks"], cfg["kinds"], Params(3, mu=cfg["mu"], sigma=cfg["sigma"], K=10 ** 9))
    c.bind(pool["last_access"], pool["queue"], np.zeros(pool["n_blocks"], np.int32), pool["ntok"], pool["ob"],
           pool["omax"], pool["valid"], pool["ref_count"], pool["parent"], pool["hash"])
    rows = []
    for k in (64, 256, 1024):
        snap = c.score_select(pool["now"], k)[2]
        casc = c.decide_cascade(pool["now"], k)
        differ = len(set(casc.tolist()) - set(snap.tolist()))
        rows.append((k, differ))
        print("tiny pool, k = %d: %d of %d cascade victims are parents promoted within the decision "
              "(not in the snapshot decision)" % (k, differ, len(casc)))
        promoted = set(casc.tolist()) - set(snap.tolist())
        assert all(pool["parent"][pool["parent"] >= 0].tolist().count(b) >= 1 for b in promoted)
    assert rows[-1][1] >= rows[0][1]


def test_what_batching_changes_on_trace_replay():
    """Balanced mix, one 36K-token cache, 4,000 requests: block hit ratio
    with snapshot decisions and with cascading ones."""
    out = {}
    for mode in ("snapshot", "cascade"):
        be = OracleBackend([0], 2250, [0, 1, 2, 2], [0, 1, 2, 3], [0.0, 0.0, 11.73, 9.19], [1, 1, 1.25, 1.34], 32, 3,
                           cascade=(mode == "cascade"))
        rd = Replay(be, 1, 2250, 1, 1024, 4)
        g = TraceGen("balanced", 1003000)
        for _ in range(4000):
            rd.step({0: g.next()})
        out[mode] = rd.summary()
        print("trace, %s decisions: %s" % (mode, {k: out[mode][k] for k in ("block_hit_ratio", "evicted",
                                                                            "decisions")}))
    assert out["snapshot"]["evicted"] > 0 and out["cascade"]["evicted"] > 0


def closure_order(c, now, k):
    """The cascade as a sort: a block can go once every cached child has
    gone, so it is eligible when valid, unreferenced and all its cached
    children are eligible; with kappa = (stage, key, id) (stage 0 for the
    evict-first queue, ordered by num_tokens) its rank is
    E(b) = max(kappa(b), E(children)), ties (which lie on one path) deepest
    first.  The first k of that order are the cascade's victims."""
    key, _ = c.keys(now)
    N = c.N
    kids = [[] for _ in range(N)]
    for b in range(N):
        if c.valid[b] and c.parent[b] >= 0:
            kids[c.parent[b]].append(b)
    memo = {}

    def info(b):  # (eligible, E, height)
        if b in memo:
            return memo[b]
        ok = bool(c.valid[b]) and c.ref_count[b] == 0
        ef = c.kind[c.queue[b]] == EVICT_FIRST
        E = (0, int(c.ntok[b]), b) if ef else (1, int(key[b]), b)
        h = 0
        for ch in kids[b]:
            o, e, hh = info(ch)
            ok = ok and o
            E = max(E, e)
            h = max(h, hh + 1)
        memo[b] = (ok, E, h)
        return memo[b]
    elig = [(info(b)[1], info(b)[2], b) for b in range(N) if info(b)[0]]
    elig.sort()
    return np.array([b for _, _, b in elig[:k]], np.int32)


def forest_cache(seed, n=80):
    rng = np.random.default_rng(seed)
    c = OracleCache(n, KINDS, Params(4, mu=[0, 0, 9.0, 0], sigma=1.2, K=1000))
    parent = np.full(n, -1, np.int32)
    for b in range(1, n):
        if rng.random() < 0.75:
            parent[b] = rng.integers(0, b)           # any earlier block: trees with several children
    la = rng.integers(0, 5000, n)
    la[rng.random(n) < 0.3] = 1234
    c.bind(la, rng.integers(0, 4, n), rng.integers(0, 5, n), rng.integers(1, 5, n), rng.integers(0, 20, n),
           np.full(n, 20), rng.random(n) < 0.9, (rng.random(n) < 0.08).astype(np.int32), parent,
           rng.integers(1, 2 ** 62, n, dtype=np.uint64))
    return c


@pytest.mark.parametrize("seed", range(12))
def test_cascade_equals_subtree_max_order(seed):
    """The order a data-parallel cascade can use (sort by the subtree maximum)
    gives exactly the sequential cascade, evict-first stage included."""
    c = forest_cache(seed)
    for k in (1, 3, 10, 40, 80):
        assert np.array_equal(closure_order(c, 6000, k), c.decide_cascade(6000, k)), k
