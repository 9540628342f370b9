"""Pins of the oracle's Algorithm 4 (online log-normal MLE, App. B) and of the
decay-power learner (App. B) against exact statistics, closed forms,
hand-built caches and the estimator's consistency on drawn samples."""
import math
import statistics

import numpy as np
import pytest

from oracle import _native as N
from oracle.policy import (EVICT_FIRST, IVL_CAP, LOGNORMAL, N_BINS, RECENCY, STRUCTURAL, OracleCache, Params,
                           sample_moments)

F32 = np.float32


@pytest.fixture(scope="module", autouse=True)
def _built(oracle_lib):
    return oracle_lib


def ulps(y, ref):
    sp = float(np.spacing(np.abs(F32(ref))))
    return abs(float(y) - float(ref)) / sp


def fp32_logs(dt):
    return [float(v) for v in N.ln(np.asarray(dt, np.float64).astype(F32))]


# ------------------------------------------------------ the sample moments
@pytest.mark.parametrize("seed", range(6))
def test_sample_moments_equal_exact_statistics(seed):
    """mu_sample and sigma_sample are the mean and population std of the fp32
    logs, to within one fp32 ulp of Python's exactly rounded statistics."""
    rng = np.random.default_rng(seed)
    n = int(rng.integers(21, 4097))
    dt = np.clip(np.round(np.exp(rng.normal(11.7, 1.3, n))), 1, 2 ** 31 - 1).astype(np.int64)
    if seed == 0:
        dt[:5] = [1, 1, 2, 2 ** 31 - 1, 3]
    xs = fp32_logs(dt)
    mu, sd = sample_moments(dt)
    assert ulps(mu, statistics.fmean(xs)) <= 1
    assert ulps(sd, statistics.pstdev(xs)) <= 1
    # and the recipe's ln keeps them within a few fp32 ulps of the fp64 logs
    lx = [math.log(float(v)) for v in dt.astype(F32)]
    assert abs(float(mu) - statistics.fmean(lx)) < 4e-6
    assert abs(float(sd) - statistics.pstdev(lx)) < 1e-5


def test_sample_moments_closed_forms():
    mu, sd = sample_moments([777] * 40)
    assert mu == F32(N.ln(np.array([777], F32))[0]) and sd == F32(0.0)
    mu, sd = sample_moments([1] * 25)                        # ln 1 = 0
    assert mu == F32(0.0) and sd == F32(0.0)
    # two-point sample: mean (ln a + ln b) / 2, population std |ln a - ln b| / 2
    a, b = 30, 24000
    mu, sd = sample_moments([a, b] * 11)
    assert abs(float(mu) - (math.log(a) + math.log(b)) / 2) < 3e-6
    assert abs(float(sd) - (math.log(b) - math.log(a)) / 2) < 3e-6    # n - 1 would give 1.0241x


# --------------------------------------------------------- caches to drive
def _ln_cache(n=64, kinds=(STRUCTURAL, LOGNORMAL, LOGNORMAL, RECENCY), learn_ln=True, learn_gamma=False, **kw):
    prm = Params(len(kinds), mu=[0, 11.7, 9.2, 0], sigma=[1, 1.25, 1.34, 1], K=4, learn_w=False,
                 learn_alpha=False, learn_ln=learn_ln, learn_gamma=learn_gamma, **kw)
    return OracleCache(n, list(kinds), prm, ghost_window=1000)


def _bind_chains(c, chains, queue, la, ob=None, omax=None):
    """Bind chains of block ids (lists) with their queues and last accesses."""
    n = c.N
    parent = np.full(n, -1, np.int32)
    valid = np.zeros(n, bool)
    for ch in chains:
        for i, b in enumerate(ch):
            valid[b] = True
            parent[b] = ch[i - 1] if i else -1
    hashes = np.arange(1, n + 1, dtype=np.uint64) * np.uint64(0x9E3779B97F4A7C15)
    z = np.zeros(n, np.int32)
    c.bind(la, queue, z, np.full(n, 16), z if ob is None else ob, z if omax is None else omax, valid, z, parent,
           hashes)
    return hashes


def test_intervals_recorded_per_request_deepest_block():
    c = _ln_cache()
    n = c.N
    queue = np.zeros(n, np.int32)
    la = np.full(n, 500, np.int32)
    # chain 0: struct 0,1 then chat (queue 1) 2,3,4; chain 1: struct 10, agent (queue 2) 11, 12
    chains = [[0, 1, 2, 3, 4], [10, 11, 12], [20, 21], [30, 31], [40, 41]]
    queue[[2, 3, 4, 21, 31]] = 1
    queue[[11, 12]] = 2
    la[[2, 3]] = 950                        # shallower chat blocks: not the recorded ones
    la[4] = 900                             # deepest chat block of chain 0
    la[12] = 400
    la[21] = 1000                           # dt = 0: nothing recorded
    la[31] = 1300                           # accessed after now: nothing recorded
    h = _bind_chains(c, chains, queue, la)
    H = lambda ids: [h[b] for b in ids]
    reqs = np.zeros((7, 6), np.uint64)
    lens = np.array([5, 3, 2, 2, 5, 2, 3], np.int32)
    reqs[0, :5] = H(chains[0])
    reqs[1, :3] = H([10, 11, 12]); reqs[1, 2] = 99            # miss at 12: deepest agent hit is 11
    reqs[2, :2] = H(chains[2])
    reqs[3, :2] = H(chains[3])
    reqs[4, :5] = H(chains[0])                                # same blocks again: same snapshot
    reqs[5, :2] = H(chains[4])                                # structural / recency only
    reqs[6, :3] = H([0, 1, 2])                                # chat block 2 is its deepest
    c.prefix_match(reqs, lens, now=1000, intervals=True)
    assert c.ivl[1] == [100, 100, 50]
    assert c.ivl[2] == [500]
    assert c.ivl[0] == [] and c.ivl[3] == []
    assert c.la[4] == 1000 and c.la[11] == 1000             # touches applied after the call
    c.prefix_match(reqs, lens, now=1100)                     # no interval flag: nothing recorded
    assert c.ivl[1] == [100, 100, 50]


def test_interval_buffer_keeps_the_newest():
    m = IVL_CAP + 10
    c = _ln_cache(n=m, kinds=(LOGNORMAL,))
    c.prm.mu = np.array([11.7], F32)
    c.prm.sigma = np.array([1.25], F32)
    h = _bind_chains(c, [[b] for b in range(m)], np.zeros(m, np.int32), np.arange(m, dtype=np.int32))
    reqs = h[:, None].copy()
    c.prefix_match(reqs, np.ones(m, np.int32), now=m + 5, touch=False, stats=False, intervals=True)
    assert c.ivl[0] == [m + 5 - r for r in range(10, m)]


def test_algorithm4_gate_ema_and_truncation():
    c = _ln_cache()
    rng = np.random.default_rng(3)
    dt = [int(v) for v in np.clip(np.round(np.exp(rng.normal(8.0, 0.9, 400))), 1, None)]
    mu0, s0 = c.prm.mu[1], c.prm.sigma[1]
    c.ivl[1] = dt[:20]
    c.feedback(force=True)
    assert c.prm.mu[1] == mu0 and c.prm.sigma[1] == s0 and c.ivl[1] == dt[:20]   # needs more than 20
    c.ivl[1] = dt[:21]
    c.feedback(force=True)
    xs = fp32_logs(dt[:21])
    want_mu = float(mu0) + 0.1 * (statistics.fmean(xs) - float(mu0))
    want_sd = float(s0) + 0.1 * (statistics.pstdev(xs) - float(s0))
    assert abs(float(c.prm.mu[1]) - want_mu) < 4e-6 and abs(float(c.prm.sigma[1]) - want_sd) < 4e-6
    assert c.ivl[1] == dt[:21]
    # 300 intervals: the update uses all of them and keeps the last 200
    mu1, s1 = float(c.prm.mu[1]), float(c.prm.sigma[1])
    c.ivl[1] = dt[:300]
    c.feedback(force=True)
    xs = fp32_logs(dt[:300])
    assert abs(float(c.prm.mu[1]) - (mu1 + 0.1 * (statistics.fmean(xs) - mu1))) < 4e-6
    assert c.ivl[1] == dt[100:300]
    # the next update sees those 200 plus what was recorded since
    mu2 = float(c.prm.mu[1])
    c.ivl[1] = c.ivl[1] + dt[300:305]
    c.feedback(force=True)
    xs = fp32_logs(dt[100:305])
    assert abs(float(c.prm.mu[1]) - (mu2 + 0.1 * (statistics.fmean(xs) - mu2))) < 4e-6
    assert c.ivl[1] == dt[105:305]
    # queue 2 had no intervals: untouched
    assert c.prm.mu[2] == F32(9.2) and c.prm.sigma[2] == F32(1.34)


def test_algorithm4_sigma_floor_and_flag():
    c = _ln_cache()
    c.prm.sigma[1] = F32(0.105)
    c.ivl[1] = [4000] * 30                                   # sigma_sample = 0
    c.feedback(force=True)
    assert c.prm.sigma[1] == F32(0.1)                        # 0.0945 floored at 0.1
    off = _ln_cache(learn_ln=False)
    off.ivl[1] = [4000] * 30
    off.feedback(force=True)
    assert off.prm.mu[1] == F32(11.7) and len(off.ivl[1]) == 30


def test_algorithm4_recovers_the_generating_lognormal():
    """Drawn from LN(mu*, sigma*), repeated updates settle near (mu*, sigma*)."""
    c = _ln_cache(kinds=(LOGNORMAL,))
    c.prm.mu = np.array([4.0], F32)
    c.prm.sigma = np.array([3.0], F32)
    rng = np.random.default_rng(11)
    mu_t, sd_t = 9.19, 1.34
    for _ in range(120):
        c.ivl[0] = c.ivl[0] + [int(v) for v in np.clip(np.round(np.exp(rng.normal(mu_t, sd_t, 60))), 1, None)]
        c.feedback(force=True)
    assert abs(float(c.prm.mu[0]) - mu_t) < 0.08
    assert abs(float(c.prm.sigma[0]) - sd_t) < 0.08


# ------------------------------------------------------ decay power (gamma)
def test_positional_bins():
    c = _ln_cache(n=8, learn_ln=False)
    c.ob[:] = [0, 1, 7, 8, 63, 64, 90, 0]
    c.omax[:] = [64, 64, 64, 64, 64, 64, 64, 0]
    assert [c.pos_bin(b) for b in range(8)] == [0, 0, 0, 1, 7, 7, 7, 0]
    c.ob[:2], c.omax[:2] = [2, 3], [3, 3]
    assert c.pos_bin(0) == 5 and c.pos_bin(1) == 7               # floor(16 / 3), the end


def _gamma_cache():
    return _ln_cache(n=8, learn_ln=False, learn_gamma=True)


def test_decay_power_worked_examples():
    c = _gamma_cache()
    c.bin_hits = [5] * N_BINS                                 # every bin's rate is 1: ratio 1
    c.feedback(force=True)
    assert abs(float(c.prm.gamma) - (1 + 0.1 * (1 / 1.1 - 1))) < 1e-6
    assert c.bin_hits == [0] * N_BINS                         # restart after an update
    c.prm.gamma = F32(1.0)
    c.bin_hits = [3, 3, 3, 3, 0, 0, 0, 0]
    c.bin_missed = [0, 0, 0, 0, 4, 4, 4, 4]                   # back rate 0: estimate 10
    c.feedback(force=True)
    assert abs(float(c.prm.gamma) - 1.9) < 1e-6
    for _ in range(30):
        c.bin_hits = [3, 3, 3, 3, 0, 0, 0, 0]
        c.bin_missed = [0, 0, 0, 0, 4, 4, 4, 4]
        c.feedback(force=True)
    assert c.prm.gamma == F32(3.0)                            # clip
    # front rates 1, 0.5, -, 0 (mean 0.5) and back 0.25, -, -, - : ratio 0.5
    c.prm.gamma = F32(1.0)
    c.bin_hits = [4, 2, 0, 0, 3, 0, 0, 0]
    c.bin_missed = [0, 2, 0, 6, 9, 0, 0, 0]
    c.feedback(force=True)
    assert abs(float(c.prm.gamma) - (1 + 0.1 * (1 / 0.6 - 1))) < 1e-6
    # back reused more than front: ratio 10, estimate 1/10.1; down to the clip
    for _ in range(40):
        c.bin_hits = [1, 0, 0, 0, 10, 10, 0, 0]
        c.bin_missed = [9, 0, 0, 0, 0, 0, 0, 0]
        c.feedback(force=True)
    assert c.prm.gamma == F32(0.3)


def test_decay_power_gates():
    c = _gamma_cache()
    c.bin_hits = [6, 5, 5, 5, 0, 0, 0, 0]                     # back half without events
    c.feedback(force=True)
    assert c.prm.gamma == F32(1.0) and c.bin_hits[0] == 6
    c.bin_hits = [0, 0, 0, 0, 5, 5, 5, 5]
    c.bin_missed = [6, 0, 0, 0, 0, 0, 0, 0]                   # front rate 0: ratio undefined
    c.feedback(force=True)
    assert c.prm.gamma == F32(1.0) and c.bin_missed[0] == 6
    c.bin_hits = [5, 5, 0, 0, 5, 5, 0, 0]                     # 20 events: not enough
    c.bin_missed = [0] * N_BINS
    c.feedback(force=True)
    assert c.prm.gamma == F32(1.0)
    c.bin_hits[7] = 1                                         # 21
    c.feedback(force=True)
    assert c.prm.gamma != F32(1.0) and c.bin_hits == [0] * N_BINS


def test_decay_power_counts_structural_hits_and_misses():
    c = _ln_cache(n=32, kinds=(STRUCTURAL, LOGNORMAL, RECENCY), learn_ln=False, learn_gamma=True)
    n = c.N
    queue = np.zeros(n, np.int32)
    queue[16:24] = 1
    queue[24:] = 2
    ob = np.zeros(n, np.int32)
    omax = np.zeros(n, np.int32)
    ob[:8], omax[:8] = np.arange(8) * 2, 15                  # bins 0 1 2 3 4 5 6 7
    ob[8:16], omax[8:16] = np.arange(8), 7                   # bins 0 1 2 3 4 5 6 8->7
    ob[16:24], omax[16:24] = np.arange(8), 7                 # log-normal queue: not counted
    chains = [list(range(0, 8)), list(range(8, 16)), list(range(16, 24)), list(range(24, 32))]
    h = _bind_chains(c, chains, queue, np.zeros(n, np.int32), ob, omax)
    reqs = np.array([h[0:8], h[0:8], h[8:16], h[16:24], h[24:32]], np.uint64)
    lens = np.array([8, 3, 8, 8, 8], np.int32)
    c.prefix_match(reqs, lens, now=10)
    assert c.bin_hits == [3, 3, 3, 2, 2, 2, 2, 2]
    # evict the two structural tails and the log-normal tail, then add them back
    dec = np.array([7, 15, 23], np.int32)
    c.commit(dec)
    for b in dec.tolist():
        c.insert([b], [h[b]], [b - 1], [20], [queue[b]], [0], [16], [ob[b]], [omax[b]])
    assert c.bin_missed == [0, 0, 0, 0, 0, 0, 0, 2]
    assert c.missed[0] == 3


def test_bins_only_while_the_learner_is_on():
    c = _ln_cache(n=16, kinds=(STRUCTURAL, RECENCY), learn_ln=False, learn_gamma=False)
    h = _bind_chains(c, [list(range(8))], np.zeros(16, np.int32), np.zeros(16, np.int32),
                     np.arange(16, dtype=np.int32), np.full(16, 7, np.int32))
    c.prefix_match(h[None, :8], [8], now=10)
    assert c.bin_hits == [0] * N_BINS and sum(c.hits) == 8
    c.commit(np.array([7], np.int32))
    c.insert([7], [h[7]], [6], [20], [0], [0], [16], [7], [7])
    assert c.bin_missed == [0] * N_BINS and c.missed[0] == 1


# ------------------------------------------- the appendix text's rule forms
def _form_cache(kinds=(EVICT_FIRST, STRUCTURAL, LOGNORMAL, RECENCY), n=64, **kw):
    prm = Params(len(kinds), K=4, learn_w=False, learn_alpha=False, learn_w_ema=True, learn_alpha_rel=True, **kw)
    return OracleCache(n, list(kinds), prm, ghost_window=1000)


def test_token_weight_ema_worked_examples():
    c = _form_cache()
    c.prm.w[:] = [2.0, 0.1, 4.99, 1.0, 1.0]
    c.evicted = [20, 0, 10, 0, 0]
    c.missed = [5, 0, 10, 0, 0]
    c.type_hits = [30, 0, 10, 0, 7]
    c.type_added = [10, 0, 0, 0, 7]
    c.feedback(force=True)
    # target 1 + 5 (5/20) + 2 (30/40) = 3.75: 0.99 * 2 + 0.01 * 3.75
    assert abs(float(c.prm.w[0]) - 2.0175) < 1e-6
    assert abs(float(c.prm.w[1]) - 0.109) < 1e-7                  # no data: target 1
    assert c.prm.w[2] == F32(5.0)                                 # target 8, clamped at 5
    assert abs(float(c.prm.w[4]) - 1.01) < 1e-6                   # r_reuse 1/2: target 2
    assert c.evicted[0] == 19 and c.missed[0] == 4 and c.type_hits[0] == 29 and c.type_added[0] == 9


def test_token_weight_ema_converges_to_its_target():
    c = _form_cache()
    c.prm.w[:] = 1.0
    for _ in range(700):
        c.evicted[:] = [100, 100, 100, 100, 100]
        c.missed[:] = [25, 0, 50, 10, 0]
        c.type_hits[:] = [90, 60, 0, 20, 2]
        c.type_added[:] = [10, 40, 100, 80, 98]
        c.feedback(force=True)
    want = [1 + 5 * 0.25 + 2 * 0.9, 1 + 2 * 0.6, 1 + 5 * 0.5, 1 + 5 * 0.1 + 2 * 0.2, 1 + 2 * 0.02]
    assert np.allclose(c.prm.w, want, atol=5e-3), (c.prm.w, want)
    assert c.prm.w[0] > c.prm.w[2] > c.prm.w[1] > c.prm.w[3] > c.prm.w[4]


def test_queue_weight_relative_efficiency_worked_examples():
    c = _form_cache()
    c.valid[:] = False
    c.valid[:60] = True
    c.queue[:] = np.repeat([0, 1, 2, 3], 16)[:64]
    c.queue[:60] = np.concatenate([np.full(10, 0), np.full(30, 1), np.full(10, 2), np.full(10, 3)])
    assert c.resident() == [10, 30, 10, 10]
    c.hits = [9, 30, 10, 0]
    c.evictions = [1, 1, 1, 1]
    c.feedback(force=True)
    # shares 30/60, 10/60, 10/60: E = 60, 60, 0, mean 40: targets 1.5, 1.5, 0
    assert abs(float(c.prm.alpha[1]) - (0.1 + 0.9 * 1.5)) < 1e-6
    assert abs(float(c.prm.alpha[2]) - (0.1 + 0.9 * 1.5)) < 1e-6
    assert c.prm.alpha[3] == F32(0.1)                             # 0.1 * 1 + 0: at the floor
    assert c.prm.alpha[0] == F32(1.0) and c.hits[0] == 9          # evict-first untouched
    assert c.hits[1:] == [0, 0, 0] and c.evictions[1:] == [0, 0, 0]
    # temperature 2: the square root of the relative efficiency
    c.prm.alpha[:] = 1.0
    c.prm.T = F32(2.0)
    c.hits = [0, 30, 10, 0]
    c.feedback(force=True)
    assert abs(float(c.prm.alpha[1]) - (0.1 + 0.9 * math.sqrt(1.5))) < 2e-6
    # equal efficiencies: every target is 1
    c.prm.alpha[:] = [1.0, 2.0, 0.5, 3.0]
    c.hits = [0, 30, 10, 10]
    c.feedback(force=True)
    assert np.allclose(c.prm.alpha[1:], [0.1 * 2.0 + 0.9, 0.1 * 0.5 + 0.9, 0.1 * 3.0 + 0.9], atol=1e-6)
    # no hits at all: nothing moves
    before = c.prm.alpha.copy()
    c.feedback(force=True)
    assert np.array_equal(before, c.prm.alpha)


def test_text_forms_count_only_when_chosen():
    c = _form_cache(kinds=(STRUCTURAL, RECENCY), n=16)
    h = _bind_chains(c, [list(range(8))], np.zeros(16, np.int32), np.zeros(16, np.int32))
    c.tau[:] = [0, 0, 1, 1, 2, 3, 3, 4] + [0] * 8
    c.prefix_match(h[None, :8], [8], now=10)
    assert c.type_hits == [2, 2, 1, 2, 1]
    c.commit(np.array([7], np.int32))
    c.insert([7], [h[7]], [6], [20], [1], [4], [16], [0], [0])
    assert c.type_added == [0, 0, 0, 0, 1] and c.resident() == [7, 1]
    off = _ln_cache(n=16, kinds=(STRUCTURAL, RECENCY), learn_ln=False)
    h = _bind_chains(off, [list(range(8))], np.zeros(16, np.int32), np.zeros(16, np.int32))
    off.prefix_match(h[None, :8], [8], now=10)
    assert off.type_hits == [0] * 5
    with pytest.raises(AssertionError):
        Params(2, learn_w=True, learn_w_ema=True)
