"""Pins of the CPU oracle against what the paper and mathematics fix.

None of these retypes the oracle's own formula: they check closed forms,
printed values, libm/mpmath accuracy bounds, monotonicity, brute force and
reductions to textbook policies (LRU).
"""
import math
import os

import numpy as np
import pytest

import oracle
from oracle import _native as N
from oracle import fp64
from oracle.policy import EVICT_FIRST, LOGNORMAL, RECENCY, STRUCTURAL, OracleCache, Params, block_type

F32 = np.float32
GOLD = os.path.join(os.path.dirname(__file__), "golden")
LN1000 = math.log(1000.0)


@pytest.fixture(scope="module", autouse=True)
def _built(oracle_lib):
    return oracle_lib


def ulps(y, ref):
    ref = np.asarray(ref, np.float64)
    sp = np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64)
    sp[sp == 0] = np.spacing(np.float32(0))
    return np.abs(np.asarray(y, np.float64) - ref) / sp


# ---------------------------------------------------------------- fp32 recipe
def test_ln_closed_forms_and_accuracy():
    assert N.ln([1.0])[0] == 0.0
    x = np.arange(1, 1 << 20, dtype=np.int64).astype(np.float32)
    y = N.ln(x)
    assert ulps(y, np.log(x.astype(np.float64))).max() <= 1.0
    assert np.all(np.diff(y) >= 0), "ln must be non-decreasing on integers"
    # (0, 1]: every float in [2^-16, 1]
    u = np.arange(np.float32(2.0 ** -16).view(np.uint32), np.float32(1).view(np.uint32) + 1, 7, dtype=np.uint32)
    r = u.view(np.float32)
    yr = N.ln(r)
    assert ulps(yr, np.log(r.astype(np.float64))).max() <= 2.0
    assert np.all(np.diff(yr) >= 0)
    # ln of powers of two is e * ln 2 to the rounding of the split constant
    for e in range(-20, 31):
        assert abs(float(N.ln([2.0 ** e])[0]) - e * math.log(2)) <= 2 * np.spacing(np.float32(abs(e) * 0.7 + 1e-30))


def test_exp_closed_forms_and_accuracy():
    assert N.exp([0.0])[0] == 1.0
    y = np.linspace(-86.0, 20.0, 400001).astype(np.float32)
    e = N.exp(y)
    ref = np.exp(y.astype(np.float64))
    assert (np.abs(e - ref) / ref).max() <= 2e-7
    assert np.all(np.diff(e) >= 0)
    assert N.exp([-87.0])[0] == 0.0 and np.isinf(N.exp([89.0])[0])


def test_erfc_against_mpmath():
    import mpmath
    assert N.erfc([0.0])[0] == 1.0
    assert N.erfc([9.0])[0] == 0.0 and N.erfc([100.0])[0] == 0.0
    x = np.concatenate([np.linspace(0, 9, 20001)[:-1], [1e-6, 1e-3, 0.4769362762044699]]).astype(np.float32)
    e = N.erfc(x).astype(np.float64)
    ref = np.array([float(mpmath.erfc(mpmath.mpf(float(v)))) for v in x])
    # published fit: fractional error < 1.2e-7; fp32 evaluation adds a few ulps
    assert (np.abs(e - ref) / ref).max() <= 5e-7
    xs = np.linspace(0, 8.99, 300001).astype(np.float32)
    assert np.all(np.diff(N.erfc(xs)) <= 0), "erfc must be non-increasing"


def test_pow01_closed_forms():
    r = np.linspace(0, 1, 1001).astype(np.float32)
    assert np.array_equal(N.pow01(r, 1.0), r)                 # gamma = 1
    assert N.pow01([0.0], 0.3)[0] == 0.0 and N.pow01([1.0], 2.7)[0] == 1.0
    rr = np.linspace(1e-4, 1, 20001).astype(np.float32)
    for g in (0.3, 0.5, 0.94, 2.0, 3.0):
        y = N.pow01(rr, g)
        ref = rr.astype(np.float64) ** g
        assert (np.abs(y - ref) / ref).max() <= 3e-6
        assert np.all(np.diff(y) >= 0)
    # squares are exact products in the reals
    assert abs(N.pow01([0.5], 2.0)[0] - 0.25) <= 2e-7


# --------------------------------------------------------------------- Eq. 1
def _golden_fits():
    rows = []
    with open(os.path.join(GOLD, "interturn_lognormal_fits.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            src, mu, sg, D, q, sec = line.split()
            rows.append((src, float(mu), float(sg), float(D), float(q), float(sec)))
    return rows


@pytest.mark.parametrize("row", _golden_fits(), ids=lambda r: "%s-q%.2f" % (r[0], r[4]))
def test_eq1_matches_printed_lognormal_fits(row):
    """Tables 3 and 5: the fitted CDF at each printed empirical percentile lies
    within the printed K-S distance of that percentile (time in ms ticks)."""
    src, mu, sg, D, q, sec = row
    dt = int(round(sec * 1000))
    p = float(N.p_lognormal([dt], mu + LN1000, sg)[0])
    assert abs((1.0 - p) - q) <= D + 0.005


def test_eq1_golden_rejects_planted_mistakes():
    """The golden check above has teeth: a dropped sqrt(2), a sign flip, or
    sigma used as a variance each fail it for some printed row."""
    rows = _golden_fits()
    def fails(fn):
        return any(abs((1 - fn(math.log(sec), mu, sg)) - q) > D + 0.005 for _, mu, sg, D, q, sec in rows)
    assert fails(lambda l, mu, s: 0.5 * math.erfc((l - mu) / s))
    assert fails(lambda l, mu, s: 0.5 * math.erfc((mu - l) / (s * math.sqrt(2))))
    assert fails(lambda l, mu, s: 0.5 * math.erfc((l - mu) / (s * s * math.sqrt(2))))
    assert not fails(lambda l, mu, s: fp64.p_lognormal(math.exp(l), mu, s))


def test_eq1_median_is_half_and_accuracy():
    for dt0 in (7, 1000, 123456, 999999):
        mu = float(N.ln([float(dt0)])[0])         # ln dt0 == mu exactly, so u = 0
        assert N.p_lognormal([dt0], mu, 1.3)[0] == np.float32(0.5)
    rng = np.random.default_rng(5)
    dt = rng.integers(1, 2 ** 24, 20000)
    for mu, sg in ((4.82 + LN1000, 1.25), (2.28 + LN1000, 1.34), (8.0, 0.3)):
        p = N.p_lognormal(dt, mu, sg).astype(np.float64)
        ref = np.array([fp64.p_lognormal(int(d), mu, sg) for d in dt])
        rel = np.abs(p - ref) / np.maximum(ref, 1e-300)
        # deep tail: the error is the fp32 rounding of ln(dt) and of u amplified
        # by the slope of ln erfc (about 2u per unit of u), plus the fit error
        u = (np.log(dt.astype(np.float64)) - mu) / (sg * math.sqrt(2))
        du = (np.abs(np.log(dt)) + abs(mu)) * 2.0 ** -23 / (sg * math.sqrt(2)) + np.abs(u) * 2.0 ** -23
        keep = ref > 1e-30
        assert np.all(rel[keep] <= 2e-6 + 2.5 * np.abs(u[keep]) * du[keep])
        full = np.arange(1, 1 << 21, dtype=np.int32)
        assert np.all(np.diff(N.p_lognormal(full, mu, sg)) <= 0), "survival is non-increasing in dt"


# --------------------------------------------------------------------- Eq. 2
def test_eq2_closed_forms():
    omax = np.arange(1, 300, dtype=np.int32)
    assert np.all(N.p_structural(np.zeros_like(omax), omax, 0.7) == 1.0)    # first block
    assert np.all(N.p_structural(omax, omax, 0.7) == 0.0)                    # last block
    assert N.p_structural([0], [0], 2.0)[0] == 1.0                            # single-block request
    ob = np.array([o // 3 for o in omax], np.int32)
    p1 = N.p_structural(ob, omax, 1.0)
    assert np.array_equal(p1, F32(1) - ob.astype(F32) / omax.astype(F32))  # gamma = 1: 1 - o_b/o_max
    for g in (0.3, 0.94, 3.0):
        ref = np.array([fp64.p_structural(int(a), int(b), g) for a, b in zip(ob, omax)])
        assert np.abs(N.p_structural(ob, omax, g) - ref).max() <= 2e-6
        row = N.p_structural(np.arange(0, 251, dtype=np.int32), np.full(251, 250, np.int32), g)
        assert np.all(np.diff(row) <= 0), "earlier blocks keep higher priority"


# --------------------------------------------------------------------- Eq. 3
def _pool(rng, n, kinds, ties=False):
    Q = len(kinds)
    c = dict(
        last_access=rng.integers(0, 1000 if ties else 1_000_000, n).astype(np.int32),
        queue=rng.integers(0, Q, n).astype(np.int32),
        tau=rng.integers(0, 5, n).astype(np.int32),
        ntok=rng.integers(1, 17, n).astype(np.int32),
        omax=rng.integers(0, 40 if ties else 250, n).astype(np.int32),
    )
    c["ob"] = (rng.random(n) * (c["omax"] + 1)).astype(np.int32).clip(0, c["omax"])
    if ties:
        c["last_access"] = (c["last_access"] // 250) * 250
        c["ob"] = (c["ob"] // 2) * 2
    return c


def _cache(rng, n, kinds, ties=False, prm=None, ref_frac=0.1, nonleaf_frac=0.3):
    f = _pool(rng, n, kinds, ties)
    prm = prm or Params(len(kinds), w=rng.uniform(0.1, 5, 5), alpha=rng.uniform(0.1, 3, len(kinds)),
                        mu=[4.82 + LN1000 if k == LOGNORMAL else 0 for k in kinds],
                        sigma=[1.25 if k == LOGNORMAL else 1 for k in kinds], gamma=0.8)
    c = OracleCache(n, kinds, prm)
    parent = np.full(n, -1, np.int32)
    nl = np.nonzero(rng.random(n) < nonleaf_frac)[0]
    leaves = np.setdiff1d(np.arange(n), nl)
    kids = rng.choice(leaves, min(len(nl), len(leaves)), replace=False)
    parent[kids] = nl[:len(kids)]
    c.bind(f["last_access"], f["queue"], f["tau"], f["ntok"], f["ob"], f["omax"],
           np.ones(n, bool), (rng.random(n) < ref_frac).astype(np.int32), parent,
           rng.integers(1, 2 ** 62, n, dtype=np.uint64))
    return c


def test_eq3_against_fp64():
    rng = np.random.default_rng(11)
    kinds = [STRUCTURAL, LOGNORMAL, RECENCY]
    c = _cache(rng, 5000, kinds)
    now = 1_000_000
    key, p = c.keys(now)
    P = key.view(np.float32).astype(np.float64)
    prm = c.prm
    for b in range(0, 5000, 7):
        q = c.queue[b]
        dt = max(now - int(c.la[b]), 0)
        if kinds[q] == LOGNORMAL:
            pr = fp64.p_lognormal(dt, float(prm.mu[q]), float(prm.sigma[q])) if dt else 1.0
        elif kinds[q] == STRUCTURAL:
            pr = fp64.p_structural(int(c.ob[b]), int(c.omax[b]), float(prm.gamma))
        else:
            pr = 1.0
        ref = fp64.priority(float(prm.alpha[q]), float(prm.w[c.tau[b]]), pr, dt)
        if ref == 0 or math.isinf(ref):
            assert P[b] == ref
        else:
            assert abs(P[b] - ref) / ref <= 3e-5, (b, P[b], ref)
    # dt = 0 is the most recent block: +inf
    c.la[0] = now
    assert np.isinf(c.keys(now)[0].view(np.float32)[0])


# ----------------------------------------------------------------- selection
def test_lru_reduction():
    """One recency queue with alpha = w = 1: P = 1/dt, and the k victims are
    exactly the k least recently used evictable blocks (ties: lower id)."""
    rng = np.random.default_rng(3)
    n, k = 20000, 500
    c = _cache(rng, n, [RECENCY], prm=Params(1, w=1.0, alpha=1.0))
    c.la[:] = rng.integers(0, 1 << 23, n)          # many equal timestamps too
    c.la[::5] = c.la[::5] // 1000 * 1000
    now = 1 << 23
    lists, key, dec = c.score_select(now, k)
    ev = np.nonzero(c.evictable())[0]
    lru = ev[np.lexsort((ev, c.la[ev]))][:k]
    assert np.array_equal(lists[0], lru)
    assert np.array_equal(dec, lru)


@pytest.mark.parametrize("seed", range(12))
def test_selection_brute_force_tiny(seed):
    """Tiny pools with forced ties: the per-queue lists equal a selection by
    repeated minimum over (key, id), the decision equals k literal calls of
    Algorithm 1's Evict(), and only evictable blocks are ever chosen."""
    rng = np.random.default_rng(seed)
    kinds = [[EVICT_FIRST, STRUCTURAL, LOGNORMAL, LOGNORMAL, RECENCY],
             [LOGNORMAL, STRUCTURAL, RECENCY],
             [STRUCTURAL, RECENCY]][seed % 3]
    n = int(rng.integers(1, 64))
    c = _cache(rng, n, kinds, ties=True)
    if seed % 4 == 0:
        c.ref_count[:] = 1                           # nothing evictable
    now = 1000
    for k in (1, 3, 17, 64):
        lists, key, dec = c.score_select(now, k)
        ev = c.evictable()
        for q in range(len(kinds)):
            pool = [b for b in range(n) if ev[b] and c.queue[b] == q]
            want = []
            while pool and len(want) < k:
                best = pool[0]
                for b in pool:
                    if (key[b], b) < (key[best], best):
                        best = b
                want.append(best)
                pool.remove(best)
            assert lists[q].tolist() == want
            assert len(lists[q]) == min(k, int(np.sum(ev & (c.queue == q))))
        assert dec.tolist() == c.evict_sequential_literal(now, k).tolist()
        assert np.all(ev[dec]) and len(set(dec.tolist())) == len(dec)


def test_selection_metamorphic():
    """Doubling every alpha (or every w) scales every P by exactly 2; shifting
    now and every last_access together leaves every dt unchanged.  Neither may
    change a victim."""
    rng = np.random.default_rng(8)
    kinds = [EVICT_FIRST, STRUCTURAL, LOGNORMAL, LOGNORMAL, RECENCY]
    c = _cache(rng, 30000, kinds)
    lists0, _, dec0 = c.score_select(1_000_000, 700)
    c.prm.alpha *= F32(2)
    lists1, _, dec1 = c.score_select(1_000_000, 700)
    c.prm.alpha /= F32(2)
    c.prm.w *= F32(4)
    lists2, _, dec2 = c.score_select(1_000_000, 700)
    c.prm.w /= F32(4)
    c.la += 12345
    lists3, _, dec3 = c.score_select(1_012_345, 700)
    for L in (lists1, lists2, lists3):
        assert all(np.array_equal(a, b) for a, b in zip(lists0, L))
    for d in (dec1, dec2, dec3):
        assert np.array_equal(dec0, d)


def test_evict_first_drains_first():
    rng = np.random.default_rng(9)
    kinds = [EVICT_FIRST, STRUCTURAL, LOGNORMAL]
    c = _cache(rng, 3000, kinds)
    n_ef = int(np.sum(c.evictable() & (c.queue == 0)))
    lists, key, dec = c.score_select(1_000_000, n_ef + 50)
    assert np.array_equal(dec[:n_ef], lists[0])
    assert np.all(c.queue[dec[n_ef:]] != 0)
    nt = c.ntok[lists[0]]
    assert np.all(np.diff(nt) >= 0)                 # smallest num_tokens first


# ---------------------------------------------------------------- block type
def test_block_type_median_token():
    assert block_type([[16, 0, 0, 0, 0]])[0] == 0
    assert block_type([[0, 0, 0, 0, 16]])[0] == 4
    assert block_type([[8, 8, 0, 0, 0]])[0] == 0    # lower median is rank 7
    assert block_type([[7, 9, 0, 0, 0]])[0] == 1
    assert block_type([[0, 8, 0, 8, 0]])[0] == 1
    assert block_type([[1, 1, 1, 1, 1]])[0] == 2    # n = 5, rank 2
    rng = np.random.default_rng(1)
    counts = rng.multinomial(16, [0.2] * 5, size=500)
    tau = block_type(counts)
    for c, t in zip(counts, tau):
        tokens = sorted(sum(([ty] * int(c[ty]) for ty in range(5)), []))
        assert tokens[(len(tokens) - 1) // 2] == t


# ------------------------------------------------------------ Classify
def test_classify_routing_cases():
    """Algorithm 1 Classify, cases worked from the queue definitions of Sec. 3.1:
    decode and CoT blocks and untemplated prefill go to the evict-first queue;
    multi-turn blocks to the chat or agentic queue; templated single-turn
    prefill to the structural queue."""
    from oracle.policy import (HINT_AGENTIC as AG, HINT_CONVERSATION as CV, HINT_DECODE as DE,
                               HINT_MULTI_TURN as MT, HINT_SHARED_PREFIX as SP, HINT_UNTEMPLATED as UT,
                               ROLE_AGENT, ROLE_CHAT, ROLE_EVICT, ROLE_STRUCT, classify_one)
    SYS, USER, TOOL, RESP, COT = range(5)
    cases = [
        (COT, MT | AG | CV | SP, ROLE_EVICT),   # chain-of-thought is never kept by queue
        (RESP, DE, ROLE_EVICT),                 # decode block of a single-turn request
        (SYS, UT, ROLE_EVICT),                  # untemplated wins over the system type
        (USER, MT | AG, ROLE_AGENT),            # agentic multi-turn history
        (TOOL, MT | AG | CV | SP, ROLE_AGENT),
        (USER, MT, ROLE_CHAT),                  # chat multi-turn history
        (SYS, CV | SP, ROLE_CHAT),              # later turn: the conversation id routes the template too
        (RESP, AG | CV, ROLE_CHAT),             # agentic but not flagged multi-turn: chat rule
        (TOOL, AG | SP, ROLE_STRUCT),           # single-turn tool-use template
        (SYS, 0, ROLE_STRUCT),                  # system prompt with no hint
        (USER, SP, ROLE_STRUCT),
        (USER, 0, ROLE_EVICT),                  # fall-through
        (TOOL, AG, ROLE_EVICT),
    ]
    for tau, hint, want in cases:
        assert classify_one(tau, hint) == want, (tau, hint, want)


def test_classify_properties_over_all_hints():
    from oracle.policy import (HINT_AGENTIC as AG, HINT_DECODE as DE, HINT_MULTI_TURN as MT,
                               HINT_UNTEMPLATED as UT, ROLE_AGENT, ROLE_EVICT, classify)
    tau = np.repeat(np.arange(5), 64)
    hint = np.tile(np.arange(64), 5)
    roles = [3, 0, 2, 1]  # a non-identity role -> queue map
    q = classify(tau, hint, roles)
    role = np.array([roles.index(x) for x in q])
    assert np.all(role[(tau == 4) | ((hint & (DE | UT)) != 0)] == ROLE_EVICT)
    assert np.all(((hint & MT) != 0)[role == ROLE_AGENT] & ((hint & AG) != 0)[role == ROLE_AGENT])
    assert set(role.tolist()) == {0, 1, 2, 3}


# ------------------------------------------------------------ learners (fp32)
def _learner_cache(kinds=(STRUCTURAL, LOGNORMAL, RECENCY)):
    return OracleCache(4, list(kinds), Params(len(kinds), w=1.0, alpha=1.0, eta=0.01, T=1.0, beta=0.1, K=1))


def test_algorithm3_worked_examples():
    c = _learner_cache()
    c.prm.w[:] = [2.0, 2.0, 4.99, 1.0, 1.0]
    c.evicted = [20, 10, 11, 0, 1000]
    c.missed = [5, 10, 11, 0, 7]
    c.feedback(force=True)
    # 2 * (1 + 0.01 * 0.25) in fp32
    assert c.prm.w[0].view(np.uint32) == 0x400051EC
    assert abs(float(c.prm.w[0]) - 2.005) < 2e-7
    assert c.evicted[0] == 19 and c.missed[0] == 4              # floor(0.99 x)
    assert c.prm.w[1] == F32(2.0) and c.evicted[1] == 9         # gate is evicted > 10
    assert c.prm.w[2] == F32(5.0)                                # clamp at 5
    assert c.evicted[4] == 990 and c.missed[4] == 6
    c.prm.w[3] = F32(0.05)
    c.evicted[3], c.missed[3] = 11, 0
    c.feedback(force=True)
    assert c.prm.w[3] == F32(0.1)                                # clamp at 0.1


def test_algorithm2_worked_examples():
    c = _learner_cache((EVICT_FIRST, STRUCTURAL, LOGNORMAL, RECENCY))
    c.hits = [9, 3, 2, 60]
    c.evictions = [9, 6, 5, 6]
    c.feedback(force=True)
    assert c.prm.alpha[0] == F32(1.0)                             # evict-first excluded
    assert c.hits[0] == 9 and c.evictions[0] == 9
    assert c.prm.alpha[1] == F32(1.05)                            # 1 + 0.1 (1.5 - 1)
    assert c.prm.alpha[2] == F32(1.0) and c.evictions[2] == 0     # gate evictions > 5
    assert c.prm.alpha[3] == F32(1.0) + F32(0.1) * F32(10.0)      # target 11 -> 2.0
    assert c.hits[1:] == [0, 0, 0]
    c.prm.alpha[3] = F32(2.9)
    c.hits[3], c.evictions[3] = 600, 6
    c.feedback(force=True)
    assert c.prm.alpha[3] == F32(3.0)                             # clamp at 3


# ---------------------------------------------------- commit / match / Add()
def _chain_cache(n=64, L=8):
    kinds = [LOGNORMAL, STRUCTURAL, RECENCY]
    c = OracleCache(n, kinds, Params(3, mu=[11.7, 0, 0], sigma=[1.25, 1, 1], K=4), ghost_window=10)
    rng = np.random.default_rng(0)
    hashes = rng.integers(1, 2 ** 62, n, dtype=np.uint64)
    parent = np.array([-1 if b % L == 0 else b - 1 for b in range(n)], np.int32)
    c.bind(rng.integers(0, 1000, n), rng.integers(0, 3, n), rng.integers(0, 5, n), np.full(n, 16),
           np.zeros(n), np.zeros(n), np.ones(n, bool), np.zeros(n), parent, hashes)
    return c, hashes.reshape(-1, L)


def test_prefix_match_brute_force():
    c, chains = _chain_cache()
    reqs = np.zeros((6, 8), np.uint64)
    lens = np.array([8, 5, 8, 0, 3, 8], np.int32)
    reqs[0] = chains[1]
    reqs[1, :5] = chains[2, :5]
    reqs[2] = chains[3]
    reqs[2, 4] = 12345                                            # break the chain at j = 4
    reqs[4, :3] = [chains[0, 0], 777, chains[0, 2]]               # later hits are ignored
    reqs[5] = chains[4]
    del c.index[int(chains[4, 6])]                                # deleting h_j gives match_len j
    m, matched = c.prefix_match(reqs, lens, now=2000)
    assert m.tolist() == [8, 5, 4, 0, 1, 6]
    keys = set(c.index)
    for r in range(6):
        j = 0
        while j < lens[r] and int(reqs[r, j]) in keys:
            j += 1
        assert j == m[r]
    assert c.la[c.index[int(chains[1, 3])]] == 2000
    assert sum(c.hits) == sum(m.tolist())


def test_commit_promotes_parent_and_ghost_feedback():
    c, chains = _chain_cache(n=16, L=4)
    c.la[:] = np.arange(16)
    now = 100
    # leaves are the chain tails 3, 7, 11, 15
    lists, key, dec = c.score_select(now, 2, commit=True)
    assert set(dec.tolist()) <= {3, 7, 11, 15}
    for b in dec:
        assert c.child_count[b - 1] == 0 and c.evictable()[b - 1]
    # re-adding an evicted hash counts one miss after eviction for its type
    b = int(dec[0])
    t = int(c.tau[b])
    c.insert([b], [c.hash[b]], [-1], [now], [c.queue[b]], [t], [16], [0], [0])
    assert c.missed[t] == 1
    c.valid[b] = False
    del c.index[int(c.hash[b])]
    c.insert([b], [c.hash[b]], [-1], [now], [c.queue[b]], [t], [16], [0], [0])
    assert c.missed[t] == 1                                       # counted once


def test_ghost_window_expiry():
    c, chains = _chain_cache(n=64, L=8)                          # W = 10
    c.la[:] = np.arange(64)
    _, _, d0 = c.score_select(1000, 4, commit=True)
    _, _, d1 = c.score_select(1000, 6, commit=True)               # 10 evictions after... not yet
    first = int(d0[0])
    assert c.ghost_live(c.ghost[int(c.hash[first])])             # 6 < W evictions after d0
    _, _, d2 = c.score_select(1000, 4, commit=True)               # now 10 after d0
    assert not c.ghost_live(c.ghost[int(c.hash[first])])
    t = int(c.tau[first])
    before = c.missed[t]
    c.insert([first], [c.hash[first]], [-1], [1000], [0], [t], [16], [0], [0])
    assert c.missed[t] == before


def test_learner_trigger_every_K_evictions():
    c, _ = _chain_cache(n=64, L=8)                               # K = 4
    c.la[:] = np.arange(64)
    c.score_select(1000, 3, commit=True)
    assert not c.pending
    c.score_select(1000, 2, commit=True)                          # 5 crosses 4
    assert c.pending and c.feedback() and not c.pending
    assert not c.feedback()


def test_reserved_hashes_never_match_and_are_refused():
    """0 and 2^64-1 mark empty and deleted index slots at the boundary: the
    oracle never indexes them, so a request hash with one ends the match, and
    Add() refuses a block carrying one (its parent gains no child)."""
    import oracle
    prm = oracle.Params(1, K=4)
    oc = oracle.OracleCache(8, [oracle.RECENCY], prm)
    tomb = 2 ** 64 - 1
    oc.insert(np.array([0, 1, 2]), np.array([11, tomb, 13], np.uint64), np.array([-1, 0, 0]), np.zeros(3, np.int32),
              np.zeros(3, np.int32), np.zeros(3, np.int32), np.full(3, 16), np.zeros(3), np.zeros(3))
    assert oc.valid.tolist()[:3] == [True, False, True]
    assert oc.child_count[0] == 1
    m, _ = oc.prefix_match(np.array([[11, 13, 0], [11, tomb, 13]], np.uint64), [3, 3], 5)
    assert m.tolist() == [2, 1]
