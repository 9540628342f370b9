"""GPU parity, tiny pool (4,096 blocks of 16 tokens, 3 queues, k = 64, 256
requests of up to 32 hashes): every step of the hot path against the oracle,
element by element, plus edge cases."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

import synth  # noqa: E402
from harness import Pair, say  # noqa: E402
from paper_2605_18825_amd import api  # noqa: E402


def tiny_pair(**over):
    cfg = synth.pool_config("tiny")
    n = over.pop("n_blocks", cfg["n_blocks"])
    pool = synth.make_pool(cfg, n_blocks=n, seed=over.pop("seed", None))
    k = over.pop("max_k", cfg["k"])
    kinds = over.pop("kinds", cfg["kinds"])
    mu = over.pop("mu", cfg["mu"][:len(kinds)] + [0.0] * max(0, len(kinds) - len(cfg["mu"])))
    sigma = over.pop("sigma", cfg["sigma"][:len(kinds)] + [1.0] * max(0, len(kinds) - len(cfg["sigma"])))
    return Pair(kinds, pool, k, mu=mu, sigma=sigma, **over), pool, cfg


@pytest.fixture
def tiny():
    p, pool, cfg = tiny_pair()
    yield p, pool, cfg
    p.close()


def test_block_types(tiny):
    p, _, _ = tiny
    p.check_tau()


@pytest.mark.parametrize("engine", ["auto", "scan", "batched", "fallback"])
def test_score_select(tiny, engine):
    p, pool, cfg = tiny
    flags = {"auto": 0, "scan": api.SS_ENGINE_SCAN, "batched": api.SS_ENGINE_BATCHED,
             "fallback": api.SS_FORCE_FALLBACK}[engine]
    say("tiny score_select engine=%s" % engine)
    for k in (64, 1, 17, 0):
        p.select(pool["now"], k, flags)
    st = p.status()
    assert set(st) <= {"SELECT_FALLBACK"}, st


def _early_stops(e, need, digits):
    """Digit steps of a most-significant-digit radix select of the `need`
    smallest of the distinct composites e where the crossing bin alone holds
    `need` elements while smaller bins hold others: a selection that stopped
    there on the bin's count alone would take too many."""
    n, rem = 0, need
    for i, (s, w) in enumerate(digits):
        d = ((e >> np.uint64(s)) & np.uint64((1 << w) - 1)).astype(np.int64)
        h = np.bincount(d, minlength=1 << w)
        cum = np.cumsum(h)
        b = int(np.searchsorted(cum, rem))
        below, cnt = int(cum[b] - h[b]), int(h[b])
        n += int(cnt == rem and below > 0 and i < len(digits) - 1)
        if below + cnt == rem:
            break
        e, rem = e[d == b], rem - below
    return n


def test_score_select_k_sweep(tiny):
    """k = 1 .. 64 on every engine: among these, some k put exactly k keys of a
    queue in the crossing bin of a digit with smaller keys below it (checked
    here for both composite layouts: (key, id) in 48 bits for the batched
    engine, 64 bits for the exact path)."""
    p, pool, cfg = tiny
    key, _ = p.oc.keys(pool["now"])
    ev = p.oc.evictable()
    layouts = {48: ([(37, 11), (26, 11), (15, 11), (4, 11), (0, 4)], 16),
               64: ([(53, 11), (42, 11), (31, 11), (20, 11), (9, 11), (0, 9)], 32)}
    for bits, (digits, sh) in layouts.items():
        hits = 0
        for q in range(p.Q):
            ids = np.nonzero(ev & (p.oc.queue == q))[0].astype(np.uint64)
            e = (key[ids].astype(np.uint64) << np.uint64(sh)) | ids
            hits += sum(_early_stops(e, k, digits) for k in range(1, 65) if k < len(ids))
        assert hits > 0, "no k in the sweep exercises the %d-bit case" % bits
    for flags in (api.SS_ENGINE_BATCHED, api.SS_ENGINE_SCAN, api.SS_FORCE_FALLBACK):
        say("tiny k sweep flags %d" % flags)
        for k in range(1, 65):
            p.select(pool["now"], k, flags)


def test_prefix_match_and_stats(tiny):
    p, pool, cfg = tiny
    R, L = synth.make_requests(pool["chains"], cfg["n_req"], cfg["req_len"], cfg["hit_frac"], 77)
    say("tiny prefix_match read-only")
    p.prefix_match(R, L, pool["now"], 0)
    say("tiny prefix_match touch+stats")
    m = p.prefix_match(R, L, pool["now"] + 5, api.PM_TOUCH | api.PM_STATS)
    assert (m > 0).mean() > 0.4
    p.check_pool()
    p.check_counters()
    # the touched blocks are now the most recent: the selection changes accordingly
    p.select(pool["now"] + 10, 64)


def test_commit_insert_feedback_cycle(tiny):
    p, pool, cfg = tiny
    now = pool["now"]
    rng = np.random.default_rng(5)
    for step in range(6):
        say("tiny cycle step %d" % step)
        lists, key, dec = p.select(now, 64, commit=True)
        p.check_pool()
        p.check_counters()
        # re-request some victims (Add() finds them in recently_evicted), refill the rest
        d = len(dec)
        re = rng.choice(d, size=min(d, 8), replace=False)
        ids = dec.astype(np.int32)
        hashes = pool["hash"][ids].copy()
        fresh = ~np.isin(np.arange(d), re)
        hashes[fresh] = rng.integers(1, 2 ** 62, int(fresh.sum()), dtype=np.uint64)
        pool["hash"][ids] = hashes
        counts = synth.pools.token_type_counts(rng, d)
        p.insert(ids, hashes, np.full(d, -1, np.int32), np.full(d, now, np.int32), rng.integers(0, 3, d),
                 counts, np.full(d, 16), rng.integers(0, 30, d), np.full(d, 30))
        p.check_pool()
        p.check_counters()
        p.feedback()
        p.check_params()
        p.check_counters()
        now += 1000
    assert sum(p.oc.missed) > 0
    assert p.oc.n_updates > 0
    assert not p.status()


def test_learners_forced_and_trigger():
    p, pool, cfg = tiny_pair(K=100, eta=0.05)
    try:
        now = pool["now"]
        for step in range(4):
            p.select(now, 64, commit=True)
            if step == 2:
                p.feedback(force=True)
            else:
                p.feedback()
            p.check_params()
            p.check_counters()
            now += 500
    finally:
        p.close()


# ------------------------------------------------------------------ edge cases
def test_ragged_pool_and_evict_first_queue():
    """A pool size that is not a multiple of 4 (scalar tail of the scan) and the
    5-queue layout with an evict-first queue and varying num_tokens."""
    kinds = [0, 1, 2, 2, 3]
    p, pool, cfg = tiny_pair(n_blocks=4099, kinds=kinds, mu=[0, 0, 11.7, 9.2, 0], sigma=[1, 1, 1.25, 1.34, 1],
                             max_k=200, gamma=0.8, w=[2.0, 1.5, 1.0, 1.0, 0.1], alpha=[1, 0.5, 2.0, 1.5, 1])
    try:
        rng = np.random.default_rng(1)
        p.oc.ntok[:] = rng.integers(1, 17, p.N)
        m = p.dp.meta.cpu().numpy().astype(np.int32) & 0xFFFF
        m = (m & ~(15 << 9)) | ((p.oc.ntok - 1) << 9)
        import torch
        p.dp.meta.copy_(torch.as_tensor(m.astype(np.int16)))
        for flags in (0, api.SS_ENGINE_SCAN, api.SS_ENGINE_BATCHED, api.SS_FORCE_FALLBACK):
            for k in (200, 5, 199):
                p.select(pool["now"], k, flags)
    finally:
        p.close()


def test_nothing_evictable_and_all_evictable():
    p, pool, cfg = tiny_pair(n_blocks=1000)
    try:
        import torch
        # everything referenced: nothing to evict
        ids = torch.arange(1000, dtype=torch.int32, device="cuda")
        api.sae_ref_blocks(p.ctx, ids, 1)
        p.oc.ref(np.arange(1000), 1)
        p.check_pool()
        for flags in (api.SS_ENGINE_SCAN, api.SS_ENGINE_BATCHED):
            p.select(pool["now"], 64, flags)
        assert int(p.out.decision_count[0]) == 0
        api.sae_ref_blocks(p.ctx, ids, -1)
        p.oc.ref(np.arange(1000), -1)
        p.check_pool()
        # k larger than every queue's evictable count takes all of them
        for flags in (api.SS_ENGINE_SCAN, api.SS_ENGINE_BATCHED):
            p.select(pool["now"], 64, flags)
    finally:
        p.close()


@pytest.mark.parametrize("n", [1, 3, 63, 65, 1025])
def test_very_small_pools(n):
    """Pools of a few blocks, every queue kind present (evict-first,
    structural with gamma != 1, two log-normal, recency): the batched
    engine's first pass then ends with short per-wave scoring lists and
    lanes past the pool, the scan's with a partial batch; every engine and
    the exact path equal the oracle for k = 1, 2 and the largest k."""
    kinds, mu, sigma = [0, 1, 2, 2, 3], [0, 0, 11.7, 9.2, 0], [1, 1, 1.25, 1.34, 1]
    cfg = synth.pool_config("tiny", kinds=kinds, mix=[0.15, 0.3, 0.2, 0.2, 0.15], mu=mu, sigma=sigma)
    pool = synth.make_pool(cfg, n_blocks=n, seed=4242 + n)
    p = Pair(kinds, pool, 64, mu=mu, sigma=sigma, gamma=0.8)
    try:
        for flags in (api.SS_ENGINE_BATCHED, api.SS_ENGINE_SCAN, api.SS_FORCE_FALLBACK):
            for k in (1, 2, 64):
                p.select(pool["now"], k, flags)
        assert p.status() in ([], ["SELECT_FALLBACK"])  # the forced exact path reports itself
    finally:
        p.close()


def test_ties_and_recent_blocks():
    """Many identical scores (same dt, type, offsets) and blocks touched at
    `now` (dt = 0, score +inf): ties go to the lower block id."""
    p, pool, cfg = tiny_pair(n_blocks=2048, max_k=512)
    try:
        import torch
        la = (pool["last_access"] // 200000) * 200000
        la[::7] = pool["now"]
        p.oc.la[:] = la
        p.dp.last_access.copy_(torch.as_tensor(la.astype(np.int32)))
        ob = pool["ob"] // 50 * 50
        p.oc.ob[:] = ob
        off = api.off_to_u32(api.pack_off(torch.as_tensor(ob.astype(np.int64)), torch.as_tensor(pool["omax"].astype(np.int64))))
        p.dp.off.copy_(off)
        for flags in (api.SS_ENGINE_SCAN, api.SS_ENGINE_BATCHED, api.SS_FORCE_FALLBACK):
            for k in (512, 300, 64):
                p.select(pool["now"], k, flags)
    finally:
        p.close()


def test_prefix_match_edge_lengths():
    p, pool, cfg = tiny_pair(n_blocks=4096)
    try:
        ch = pool["chains"]
        R = np.zeros((6, 130), np.uint64)
        L = np.array([0, 1, 64, 65, 130, 32], np.int32)
        R[1, 0] = ch[0, 0]
        R[2, :32] = ch[1]
        R[2, 32:64] = ch[2]                 # another chain: every hash is still indexed, match = 64
        R[3, :32] = ch[3]
        R[3, 32:65] = 12345
        R[4, :] = 999
        R[4, :32] = ch[4]
        R[5, :32] = ch[5]
        p.prefix_match(R, L, pool["now"], api.PM_STATS | api.PM_TOUCH)
        p.check_counters()
    finally:
        p.close()


def test_reserved_hashes():
    """The reserved hash values 0 and 2^64-1 (empty and deleted index slots)
    never match, even where evictions left deleted slots behind, and Add()
    refuses a block that carries one (its parent gains no child)."""
    p, pool, cfg = tiny_pair(n_blocks=4096)
    try:
        now = pool["now"]
        _, _, dec = p.select(now, 64, commit=True)        # leaves deleted slots in the index
        ch = pool["chains"]
        tomb, empty = np.uint64(2 ** 64 - 1), np.uint64(0)
        R = np.zeros((4, 32), np.uint64)
        L = np.array([32, 32, 32, 1], np.int32)
        R[0] = ch[0]
        R[0, 0] = tomb
        R[1] = ch[1]
        R[1, 5] = tomb
        R[2] = ch[2]
        R[2, 3] = empty
        R[3, 0] = empty
        m = p.prefix_match(R, L, now + 1, api.PM_STATS | api.PM_TOUCH)
        assert m[0] == 0 and m[3] == 0 and m[1] <= 5 and m[2] <= 3
        ids = dec[:3]
        live = np.nonzero(p.oc.valid)[0]
        par = np.array([-1, live[0], live[1]], np.int32)   # cached parents
        hashes = np.array([tomb, empty, np.uint64(0x1234567)], np.uint64)
        counts = np.zeros((3, 5), np.uint8)
        counts[:, 1] = 16
        p.insert(ids, hashes, par, np.full(3, now + 2, np.int32), np.array([0, 1, 2]), counts,
                 np.full(3, 16, np.int32), np.zeros(3, np.int32), np.zeros(3, np.int32))
        assert "BAD_HASH" in p.status()
        p.check_pool()
        p.check_counters()
        assert not p.oc.valid[ids[0]] and not p.oc.valid[ids[1]] and p.oc.valid[ids[2]]
        p.select(now + 3, 64, commit=True)
    finally:
        p.close()
