"""GPU parity of cascading decisions (SAE_SS_CASCADE: Algorithm 1's Evict()
one victim at a time, a parent evictable once its last cached child is taken)
against the oracle's sequential cascade, through the C ABI: the synthetic
pool with both engines, commit cycles, deep chains and shared roots (many
rounds, the touched-block list overflowing into a full reset), and the
argument checks."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

import synth  # noqa: E402
from harness import Pair, say  # noqa: E402
from paper_2605_18825_amd import api  # noqa: E402

C = api.SS_CASCADE


def tiny(n=4096, seed=None, max_k=1024, kinds=None):
    cfg = synth.pool_config("tiny")
    pool = synth.make_pool(cfg, n_blocks=n, seed=seed)
    kinds = kinds or cfg["kinds"]
    mu = (cfg["mu"] + [0.0] * 8)[:len(kinds)]
    sigma = (cfg["sigma"] + [1.0] * 8)[:len(kinds)]
    return Pair(kinds, pool, max_k, mu=mu, sigma=sigma), pool


@pytest.mark.parametrize("engine", [api.SS_ENGINE_SCAN, api.SS_ENGINE_BATCHED])
def test_cascade_decisions_synthetic_pool(engine):
    p, pool = tiny()
    try:
        for k in (64, 256, 1024, 1, 0):
            say("cascade: engine %d k %d" % (engine, k))
            p.select(pool["now"], k, engine | C)
        assert not p.status()
    finally:
        p.close()


def test_cascade_commit_cycles():
    p, pool = tiny(max_k=512)
    try:
        now = pool["now"]
        rng = np.random.default_rng(9)
        for step in range(5):
            say("cascade: cycle %d" % step)
            lists, key, dec = p.select(now, 512, C, commit=True)
            p.check_pool()
            p.check_counters()
            d = len(dec)
            ids = dec.astype(np.int32)
            hashes = rng.integers(1, 2 ** 62, d, dtype=np.uint64)
            counts = synth.pools.token_type_counts(rng, d)
            p.insert(ids, hashes, np.full(d, -1, np.int32), np.full(d, now, np.int32), rng.integers(0, 3, d), counts,
                     np.full(d, 16), np.zeros(d, np.int32), np.full(d, 30))
            p.feedback()
            p.check_params()
            now += 700
        assert not p.status()
    finally:
        p.close()


def chain_pool(n_chains, depth, fan, seed):
    """Chains under shared roots: root r has `fan` chains of `depth` blocks;
    the older a block, the closer to the root, so whole chains cascade."""
    rng = np.random.default_rng(seed)
    per = 1 + fan * depth
    n = n_chains * per
    cfg = synth.pool_config("tiny")
    pool = synth.make_pool(cfg, n_blocks=n, seed=seed)
    parent = np.full(n, -1, np.int32)
    la = np.zeros(n, np.int32)
    for c in range(n_chains):
        r = c * per
        la[r] = rng.integers(0, 1000)
        for f in range(fan):
            prev = r
            for d in range(depth):
                b = r + 1 + f * depth + d
                parent[b] = prev
                la[b] = la[prev] + rng.integers(0, 3000)
                prev = b
    pool["parent"] = parent
    pool["last_access"] = la
    pool["ref_count"] = (rng.random(n) < 0.02).astype(np.int32)
    pool["valid"] = np.ones(n, bool)
    return pool


@pytest.mark.parametrize("max_k,k", [(256, 256), (16, 16), (4096, 3000)])
def test_cascade_deep_chains_and_shared_roots(max_k, k):
    pool = chain_pool(24, 40, 3, 77 + max_k)
    cfg = synth.pool_config("tiny")
    p = Pair(cfg["kinds"], pool, max_k, mu=cfg["mu"], sigma=cfg["sigma"])
    try:
        now = int(pool["last_access"].max()) + 10
        for flags in (api.SS_ENGINE_SCAN | C, api.SS_ENGINE_BATCHED | C):
            say("cascade: chains max_k %d k %d flags %d" % (max_k, k, flags))
            lists, key, dec = p.select(now, k, flags)
        lists, key, dec = p.select(now, k, api.SS_ENGINE_SCAN | C, commit=True)
        p.check_pool()
        p.select(now + 50, k, api.SS_ENGINE_SCAN | C)  # the per-block scratch was reset
        assert not p.status()
    finally:
        p.close()


def test_cascade_argument_checks():
    cfg = synth.pool_config("tiny")
    pool = synth.make_pool(cfg, n_blocks=1024)
    p = Pair(cfg["kinds"], pool, 8192, mu=cfg["mu"], sigma=cfg["sigma"])
    try:
        with pytest.raises(api.SaeError, match="max_k <= 4096"):
            p.out.run(p.ctx, pool["now"], 64, C)
    finally:
        p.close()
