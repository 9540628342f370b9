"""GPU parity of Algorithm 4 (online log-normal MLE) and of the decay-power
learner, through the C ABI: the intervals each prefix match records, the
interval buffers, the positional-bin counters, and mu / sigma / gamma after
every update, bit for bit against the oracle."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

import synth  # noqa: E402
from harness import Pair, say  # noqa: E402
from paper_2605_18825_amd import api  # noqa: E402

ALL = api.LEARN_TOKEN_WEIGHTS | api.LEARN_QUEUE_WEIGHTS | api.LEARN_LOGNORMAL | api.LEARN_DECAY_POWER
# the appendix text's token and queue rules in place of Algorithms 3 and 2
TEXT = api.LEARN_TOKEN_EMA | api.LEARN_QUEUE_REL | api.LEARN_LOGNORMAL | api.LEARN_DECAY_POWER
FLAGS = api.PM_TOUCH | api.PM_STATS | api.PM_INTERVALS


def five_queue_pair(n_blocks, seed, max_requests, learn=ALL, **over):
    """The 5-queue layout (evict-first, structural, chat, agent, default)."""
    cfg = synth.pool_config("large")
    pool = synth.make_pool(cfg, n_blocks=n_blocks, seed=seed)
    p = Pair(cfg["kinds"], pool, over.pop("max_k", 256), mu=cfg["mu"], sigma=cfg["sigma"], learn=learn,
             max_requests=max_requests, **over)
    return p, pool, cfg


def long_requests(chains, n, rng):
    """Requests made of whole chains back to back: every hash is indexed, so
    the match runs over several 64-hash chunks (up to the length)."""
    L = chains.shape[1]
    lens = np.array([3 * L, 2 * L + 5, L + 64, 64, 65, 1][:n], np.int32)
    R = np.zeros((len(lens), 3 * L), np.uint64)
    for r, ln in enumerate(lens):
        cs = rng.integers(0, chains.shape[0], 3)
        R[r] = np.concatenate([chains[c] for c in cs])
        R[r, ln:] = 0
    return R, lens


def test_intervals_recorded_like_the_oracle():
    p, pool, cfg = five_queue_pair(8192, 4101, 2048)
    try:
        rng = np.random.default_rng(1)
        sel = rng.random(p.N)
        la = pool["last_access"].copy()
        la[sel < 0.05] = pool["now"]                              # dt = 0: not recorded
        la[(sel >= 0.05) & (sel < 0.08)] = pool["now"] + 50        # in the future: not recorded
        p.oc.la[:] = la
        p.dp.last_access.copy_(torch.as_tensor(la.astype(np.int32)))
        R, L = synth.make_requests(pool["chains"], 1024, 160, 0.7, 5)
        say("learners: intervals, 1024 requests")
        p.prefix_match(R, L, pool["now"], FLAGS)
        p.check_intervals()
        p.check_pool()
        p.check_counters()
        assert 20 < len(p.oc.ivl[2]) and 20 < len(p.oc.ivl[3])
        say("learners: intervals, whole-chain requests, no touch")
        R2, L2 = long_requests(pool["chains"], 6, rng)
        p.prefix_match(R2, L2, pool["now"] + 777, api.PM_INTERVALS)
        p.check_intervals()
        p.check_pool()
        say("learners: intervals with stats only")
        p.prefix_match(R, L, pool["now"] + 1500, api.PM_STATS | api.PM_INTERVALS)
        p.check_intervals()
        p.check_counters()
    finally:
        p.close()


def test_interval_buffer_cap():
    """One call records more than the buffer holds: the newest 4,096 stay, in
    request order, and the update uses exactly those."""
    p, pool, cfg = five_queue_pair(8192, 4102, 6000)
    try:
        ln_blocks = np.nonzero(pool["queue"] == 2)[0]
        rng = np.random.default_rng(2)
        pick = rng.choice(ln_blocks, size=min(len(ln_blocks), 2600), replace=False)
        ids = np.concatenate([pick, pick])                         # each block asked twice
        R = pool["hash"][ids][:, None].copy()
        L = np.ones(len(ids), np.int32)
        assert len(ids) > api.IVL_CAP
        say("learners: %d one-block requests" % len(ids))
        p.prefix_match(R, L, pool["now"], FLAGS)
        p.check_intervals()
        assert len(p.oc.ivl[2]) == api.IVL_CAP
        p.feedback(force=True)
        p.check_params()
        p.check_intervals()
        assert len(p.oc.ivl[2]) == 200
    finally:
        p.close()


@pytest.mark.parametrize("rules", ["algorithms", "text"])
def test_learning_cycle_all_learners(rules):
    """Prefix matches, decisions with commit, re-added victims and the
    learners every K evictions: all parameters, counters and buffers agree
    after every step.  `text`: the appendix text's token and queue rules from
    the paper's initial token weights."""
    if rules == "text":
        p, pool, cfg = five_queue_pair(8192, 4105, 512, learn=TEXT, K=200, w=list(api.PAPER_INIT_W), T=2.0)
    else:
        p, pool, cfg = five_queue_pair(8192, 4103, 512, K=200)
    try:
        rng = np.random.default_rng(3)
        now = pool["now"]
        gamma0 = float(p.prm.gamma)
        for step in range(10):
            say("learners: %s cycle step %d" % (rules, step))
            R, L = synth.make_requests(pool["chains"], 512, 48, 0.6, 100 + step)
            p.prefix_match(R, L, now, FLAGS)
            lists, key, dec = p.select(now, 256, commit=True)
            d = len(dec)
            ids = dec.astype(np.int32)
            # half the victims come back (misses after eviction), the rest are new content
            back = rng.random(d) < 0.5
            hashes = pool["hash"][ids].copy()
            hashes[~back] = rng.integers(1, 2 ** 62, int((~back).sum()), dtype=np.uint64)
            pool["hash"][ids] = hashes
            counts = synth.pools.token_type_counts(rng, d)
            queue = p.oc.queue[ids].copy()
            p.insert(ids, hashes, np.full(d, -1, np.int32), np.full(d, now, np.int32), queue, counts,
                     np.full(d, 16), p.oc.ob[ids].copy(), p.oc.omax[ids].copy())
            p.feedback()
            p.check_params()
            p.check_counters()
            p.check_intervals()
            now += 997
        assert p.oc.n_updates >= 5
        assert p.prm.mu[2] != np.float32(cfg["mu"][2]) and p.prm.mu[3] != np.float32(cfg["mu"][3])
        assert float(p.prm.gamma) != gamma0
        p.check_pool()
        assert not p.status()
    finally:
        p.close()


def test_interval_argument_errors():
    p, pool, cfg = five_queue_pair(1024, 4104, 8)
    try:
        R = torch.as_tensor(pool["hash"][:16].view(np.int64).reshape(16, 1)).cuda()
        L = torch.ones(16, dtype=torch.int32, device="cuda")
        ml = torch.zeros(16, dtype=torch.int32, device="cuda")
        mid = torch.zeros((16, 1), dtype=torch.int32, device="cuda")
        with pytest.raises(api.SaeError, match="matched_ids"):
            api.sae_prefix_match(p.ctx, R[:8], L[:8], 5, api.PM_INTERVALS, ml[:8])
        with pytest.raises(api.SaeError, match="max_requests"):
            api.sae_prefix_match(p.ctx, R, L, 5, api.PM_INTERVALS, ml, matched_ids=mid)
        with pytest.raises(api.SaeError, match="log-normal"):
            api.sae_get_intervals(p.ctx, 0, 1)
        with pytest.raises(api.SaeError, match="token-weight rule"):
            api.sae_set_params(p.ctx, 0, api.make_params(5, learn=api.LEARN_TOKEN_WEIGHTS | api.LEARN_TOKEN_EMA))
        with pytest.raises(api.SaeError, match="queue-weight rule"):
            api.sae_set_params(p.ctx, 0, api.make_params(5, learn=api.LEARN_QUEUE_WEIGHTS | api.LEARN_QUEUE_REL))
        assert api.sae_get_intervals(p.ctx, 0, 2) == []
        assert not p.status()
    finally:
        p.close()
