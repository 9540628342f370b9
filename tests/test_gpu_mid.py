"""GPU parity, mid pool (262,144 blocks, 3 queues, k = 1,024): 64 back-to-back
decisions, each committed, followed by a prefix-match batch that re-requests
5 % of the victims, Add() of those victims and of fresh blocks into the other
freed slots, and a feedback update.  Every decision, counter, learned weight
and pool bit is compared with the oracle after every cycle."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

import synth  # noqa: E402
from harness import Pair, say  # noqa: E402
from paper_2605_18825_amd import api  # noqa: E402


def run_cycles(n_cycles, n_blocks=None, check_every=1):
    cfg = synth.pool_config("mid")
    pool = synth.make_pool(cfg, n_blocks=n_blocks)
    N, k = pool["n_blocks"], cfg["k"]
    p = Pair(cfg["kinds"], pool, k, mu=cfg["mu"], sigma=cfg["sigma"], K=k)
    rng = np.random.default_rng(cfg["seed"] + 7)
    now = pool["now"]
    n_re = int(round(cfg["rerequest"] * k))
    try:
        for d in range(n_cycles):
            say("mid cycle %d" % d)
            lists, key, dec = p.select(now, k, commit=True)
            nd = len(dec)
            re = np.sort(rng.choice(nd, size=min(n_re, nd), replace=False))
            # requests: fresh chain prefixes plus one single-hash request per re-requested victim
            R, L = synth.make_requests(pool["chains"], cfg["n_req"], cfg["req_len"], cfg["hit_frac"], rng)
            R2 = np.zeros((len(re), R.shape[1]), np.uint64)
            R2[:, 0] = pool["hash"][dec[re]]
            R = np.concatenate([R, R2])
            L = np.concatenate([L, np.ones(len(re), np.int32)])
            p.prefix_match(R, L, now + 1, api.PM_TOUCH | api.PM_STATS)
            # Add(): re-requested victims keep their features; other slots get fresh blocks
            ids = dec.astype(np.int32)
            hashes = pool["hash"][ids].copy()
            fresh = np.ones(nd, bool)
            fresh[re] = False
            hashes[fresh] = synth.pools._fix_reserved(rng.integers(1, 2 ** 63, int(fresh.sum()), dtype=np.uint64))
            pool["hash"][ids] = hashes
            counts = synth.pools.token_type_counts(rng, nd)
            counts[~fresh] = pool["counts"][ids[~fresh]]
            pool["counts"][ids] = counts
            queue = np.where(fresh, rng.choice(3, size=nd, p=cfg["mix"]), p.oc.queue[ids]).astype(np.int32)
            omax = np.where(fresh, rng.integers(31, 251, nd), p.oc.omax[ids]).astype(np.int32)
            ob = np.where(fresh, (rng.random(nd) * (omax + 1)).astype(np.int32).clip(0, omax), p.oc.ob[ids]).astype(np.int32)
            p.insert(ids, hashes, np.full(nd, -1, np.int32), np.full(nd, now + 1, np.int32), queue, counts,
                     np.full(nd, 16, np.int32), ob, omax)
            fired = p.feedback()
            if d % check_every == 0 or d == n_cycles - 1:
                p.check_counters()
                p.check_params()
                p.check_pool()
            now += 1000
        assert sum(p.oc.missed) > 0 and p.oc.n_updates == n_cycles
        st = p.status()
        assert set(st) <= {"SELECT_FALLBACK"}, st
        return p
    finally:
        p.close()


def test_mid_64_decisions():
    run_cycles(64, check_every=4)
