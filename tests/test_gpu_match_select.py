"""GPU parity of sae_match_select: a prefix match and a decision in one call,
the selection's sampling and bounds sharing the prefix match's launch.

 * Mid pool (262,144 blocks, 3 queues, k = 1,024), 16 serving cycles: a
   prefix-match batch (fresh chain prefixes plus re-requests of the previous
   decision's victims) with touch and statistics and the committed decision
   in one call, Add() into the freed slots, feedback; every match length,
   matched id, list, score bit, decision entry, counter, learned parameter and
   pool bit equals the oracle's (its prefix match, then its selection).
 * The same with every learner on and Algorithm 4's intervals recorded.
 * Edge cases on the pool-scan engine: no requests, request counts that fill
   no whole workgroup, lengths 0 / 1 / 65 / 130, the cascading decision, the
   forced exact path, k = 1, the match at an earlier time than the
   selection.
 * Four instances (k per instance, one of them 0), 3,500 requests, with and
   without Algorithm 4's interval recording, against a second context
   driven by sae_prefix_match and sae_score_select: identical bit for bit,
   interval buffers included.
 * 20,000 requests on one instance: 64 per prefix-match workgroup (the
   most), more workgroups than the device holds at once, so that
   prefix-match and bound workgroups start late; identical to the two
   calls.
 * A context on the batched engine (the call runs the two halves in turn).
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

import synth  # noqa: E402
from harness import Pair, say, u64  # noqa: E402
from paper_2605_18825_amd import api  # noqa: E402
from paper_2605_18825_amd.pool import DevicePool, SelectBuffers  # noqa: E402

PM = api.PM_TOUCH | api.PM_STATS


def cycle_requests(pool, cfg, rng, evicted, n_re):
    """Fresh chain prefixes plus one single-hash request per re-requested
    victim (hashes `evicted` of the previous decision); also returns the
    re-requested hashes."""
    R, L = synth.make_requests(pool["chains"], cfg["n_req"], cfg["req_len"], cfg["hit_frac"], rng)
    re_hashes = np.zeros(0, np.uint64)
    if len(evicted):
        re_hashes = rng.choice(evicted, size=min(n_re, len(evicted)), replace=False)
        R2 = np.zeros((len(re_hashes), R.shape[1]), np.uint64)
        R2[:, 0] = re_hashes
        R = np.concatenate([R, R2])
        L = np.concatenate([L, np.ones(len(re_hashes), np.int32)])
    return R, L, re_hashes


def add_fresh(p, pool, cfg, rng, dec, now, re_hashes):
    """Add() into the slots a decision freed (both sides): the re-requested
    victims come back under their old hashes (misses after eviction), the
    other slots get fresh blocks."""
    nd = len(dec)
    if nd == 0:
        return
    ids = dec.astype(np.int32)
    hashes = synth.pools._fix_reserved(rng.integers(1, 2 ** 63, nd, dtype=np.uint64))
    m = min(nd, len(re_hashes))
    hashes[:m] = re_hashes[:m]
    pool["hash"][ids] = hashes
    counts = synth.pools.token_type_counts(rng, nd)
    queue = rng.choice(len(cfg["kinds"]), size=nd, p=cfg["mix"]).astype(np.int32)
    omax = rng.integers(31, 251, nd).astype(np.int32)
    ob = (rng.random(nd) * (omax + 1)).astype(np.int32).clip(0, omax)
    p.insert(ids, hashes, np.full(nd, -1, np.int32), np.full(nd, now, np.int32), queue, counts,
             np.full(nd, 16, np.int32), ob, omax)


def serve_cycles(n_cycles, learn, pm_flags, label):
    cfg = synth.pool_config("mid")
    pool = synth.make_pool(cfg)
    k = cfg["k"]
    max_req = cfg["n_req"] + k
    p = Pair(cfg["kinds"], pool, k, mu=cfg["mu"], sigma=cfg["sigma"], K=k, learn=learn, max_requests=max_req)
    rng = np.random.default_rng(cfg["seed"] + 31)
    now = pool["now"]
    n_re = int(round(cfg["rerequest"] * k))
    evicted = np.zeros(0, np.uint64)
    try:
        for d in range(n_cycles):
            R, L, re_hashes = cycle_requests(pool, cfg, rng, evicted, n_re)
            om, dec = p.match_select(R, L, now, pm_flags, now, k, commit=True)
            evicted = pool["hash"][dec].copy()
            add_fresh(p, pool, cfg, rng, dec, now + 1, re_hashes)
            p.feedback()
            p.check_counters()
            p.check_params()
            p.check_pool()
            if pm_flags & api.PM_INTERVALS:
                p.check_intervals()
            say("%s: cycle %d equal (%d victims, %d blocks matched)" % (label, d, len(dec), int(om.sum())))
            now += 1000
        assert sum(p.oc.missed) > 0
        st = p.status()
        assert set(st) <= {"SELECT_FALLBACK"}, st
    finally:
        p.close()


def test_mid_pool_serving_cycles():
    serve_cycles(16, 3, PM, "match+select mid")


def test_mid_pool_every_learner_with_intervals():
    serve_cycles(8, 15, PM | api.PM_INTERVALS, "match+select mid, all learners")


def test_edge_cases_on_the_scan_engine():
    cfg = synth.pool_config("tiny")
    N = 20000
    pool = synth.make_pool(cfg, n_blocks=N, seed=77)
    k = 64
    p = Pair(cfg["kinds"], pool, k, mu=cfg["mu"], sigma=cfg["sigma"], K=k)
    rng = np.random.default_rng(5)
    now = pool["now"]
    try:
        R0, L0 = synth.make_requests(pool["chains"], 40, 130, 0.8, rng)
        cases = [
            ("no requests", R0[:0], L0[:0], 0),
            ("one request", R0[:1], L0[:1], 0),
            ("15 requests", R0[:15], L0[:15], 0),
            ("17 requests", R0[:17], L0[:17], 0),
            ("lengths 0/1/65/130", R0[:4], np.array([0, 1, 65, 130], np.int32), 0),
            ("cascade", R0[:20], L0[:20], api.SS_CASCADE),
            ("forced exact path", R0[:20], L0[:20], api.SS_FORCE_FALLBACK),
            ("40 requests, commit", R0, L0, api.SS_COMMIT),
        ]
        for name, R, L, fl in cases:
            say("edge: %s" % name)
            p.match_select(R, L, now, PM, now, k, flags=fl | api.SS_ENGINE_SCAN)
            p.check_counters()
            p.check_pool()
            now += 100
        say("edge: k = 1")
        p.match_select(R0[:8], L0[:8], now, PM, now, 1, flags=api.SS_ENGINE_SCAN | api.SS_COMMIT)
        p.check_counters()
        p.check_pool()
        now += 100
        say("edge: the match 40 ticks before the selection")
        p.match_select(R0[20:], L0[20:], now - 40, PM, now, k, flags=api.SS_ENGINE_SCAN | api.SS_COMMIT)
        p.check_counters()
        p.check_pool()
        assert set(p.status()) <= {"SELECT_FALLBACK"}
    finally:
        p.close()


class Ctx:
    """A context of n_inst instances filled from `pools`."""

    def __init__(self, pools, cfg, k, max_req):
        self.n_inst, self.Q = len(pools), len(cfg["kinds"])
        self.kinds = cfg["kinds"]
        self.ctx = api.sae_create(self.n_inst, pools[0]["n_blocks"], cfg["kinds"], max_k=k, max_requests=max_req)
        self.dp = DevicePool(self.n_inst, pools[0]["n_blocks"])
        for i, pl in enumerate(pools):
            self.dp.fill_instance(i, pl)
        self.dp.bind(self.ctx)
        api.sae_index_build(self.ctx)
        api.sae_set_params(self.ctx, -1, api.make_params(self.Q, mu=cfg["mu"], sigma=cfg["sigma"], K=k, learn=3))
        self.out = SelectBuffers(self.n_inst, self.Q, k)

    def snapshot(self, ml, mid):
        torch.cuda.synchronize()
        snap = {f: getattr(self.dp, f).cpu().numpy().copy() for f in
                ("last_access", "meta", "child_count", "access_count")}
        for f in ("victims", "count", "decision", "decision_count"):
            snap[f] = getattr(self.out, f).cpu().numpy().copy()
        snap["scores"] = self.out.scores.cpu().numpy().view(np.uint32).copy()
        snap["ml"], snap["mid"] = ml.cpu().numpy().copy(), mid.cpu().numpy().copy()
        for i in range(self.n_inst):
            c = api.sae_get_counters(self.ctx, i)
            snap["c%d" % i] = np.array(list(c.evicted) + list(c.missed) + list(c.hits) + list(c.evictions) +
                                       [c.eviction_count], np.int64)
            for q in range(self.Q):
                if self.kinds[q] == api.KIND_LOGNORMAL:
                    snap["ivl%d.%d" % (i, q)] = np.array(api.sae_get_intervals(self.ctx, i, q), np.int32)
        return snap


@pytest.mark.parametrize("pm_flags", [PM, PM | api.PM_INTERVALS], ids=["touch-stats", "with-intervals"])
def test_four_instances_equal_the_two_calls(pm_flags):
    cfg = synth.pool_config("tiny")
    N, k, n_inst = 40000, 64, 4
    pools = [synth.make_pool(cfg, n_blocks=N, seed=900 + i) for i in range(n_inst)]
    a, b = Ctx(pools, cfg, k, 3500), Ctx(pools, cfg, k, 3500)
    rng = np.random.default_rng(11)
    now = max(pl["now"] for pl in pools)
    kpi = torch.tensor([k, 17, 0, 1], dtype=torch.int32, device="cuda")
    try:
        for cyc in range(6):
            # 3,500 requests over four instances: prefix-match workgroups of about 33 requests each
            R, L = synth.make_requests(pools[0]["chains"], 3500, cfg["req_len"], cfg["hit_frac"], rng)
            inst = rng.integers(0, n_inst, len(L)).astype(np.int32)
            for j in range(len(L)):  # a hit request follows a chain of its own instance
                if inst[j]:
                    R2, _ = synth.make_requests(pools[inst[j]]["chains"], 1, cfg["req_len"], cfg["hit_frac"], rng)
                    R[j, :L[j]] = R2[0, :L[j]]
            hd = torch.as_tensor(u64(R).view(np.int64)).cuda()
            ld = torch.as_tensor(L).cuda()
            idev = torch.as_tensor(inst).cuda()
            bufs = []
            for c in (a, b):
                bufs.append((torch.full((len(L),), -7, dtype=torch.int32, device="cuda"),
                             torch.full(hd.shape, -7, dtype=torch.int32, device="cuda")))
            (ml_a, mid_a), (ml_b, mid_b) = bufs
            api.sae_prefix_match(a.ctx, hd, ld, now, pm_flags, ml_a, matched_ids=mid_a, inst=idev)
            a.out.run(a.ctx, now, k, api.SS_COMMIT | api.SS_ENGINE_SCAN, k_per_inst=kpi)
            b.out.run_after_match(b.ctx, hd, ld, now, pm_flags, ml_b, now, k, api.SS_COMMIT | api.SS_ENGINE_SCAN,
                                  matched_ids=mid_b, inst=idev, k_per_inst=kpi)
            sa, sb = a.snapshot(ml_a, mid_a), b.snapshot(ml_b, mid_b)
            for key in sa:
                if not np.array_equal(sa[key], sb[key]):
                    bad = np.argwhere(sa[key] != sb[key])[:5].tolist()
                    raise AssertionError("cycle %d: %s differs at %s" % (cyc, key, bad))
            assert int(sa["decision_count"].sum()) > 0
            say("four instances: cycle %d identical (%d victims)" % (cyc, int(sa["decision_count"].sum())))
            for c in (a, b):
                api.sae_feedback_update(c.ctx, 0)
            now += 1000
    finally:
        api.sae_destroy(a.ctx)
        api.sae_destroy(b.ctx)


def test_more_workgroups_than_the_device_holds():
    cfg = synth.pool_config("mid")
    pool = synth.make_pool(cfg, n_blocks=65536, seed=31)
    k = 256
    a, b = Ctx([pool], cfg, k, 0), Ctx([pool], cfg, k, 0)
    rng = np.random.default_rng(12)
    now = pool["now"]
    try:
        for cyc in range(3):
            R, L = synth.make_requests(pool["chains"], 20000, 24, cfg["hit_frac"], rng)
            hd = torch.as_tensor(u64(R).view(np.int64)).cuda()
            ld = torch.as_tensor(L).cuda()
            out = []
            for c in (a, b):
                out.append((torch.full((len(L),), -7, dtype=torch.int32, device="cuda"),
                            torch.full(hd.shape, -7, dtype=torch.int32, device="cuda")))
            (ml_a, mid_a), (ml_b, mid_b) = out
            api.sae_prefix_match(a.ctx, hd, ld, now, PM, ml_a, matched_ids=mid_a)
            a.out.run(a.ctx, now, k, api.SS_COMMIT | api.SS_ENGINE_SCAN)
            b.out.run_after_match(b.ctx, hd, ld, now, PM, ml_b, now, k, api.SS_COMMIT | api.SS_ENGINE_SCAN,
                                  matched_ids=mid_b)
            sa, sb = a.snapshot(ml_a, mid_a), b.snapshot(ml_b, mid_b)
            for key in sa:
                if not np.array_equal(sa[key], sb[key]):
                    bad = np.argwhere(sa[key] != sb[key])[:5].tolist()
                    raise AssertionError("cycle %d: %s differs at %s" % (cyc, key, bad))
            assert int(sa["ml"].sum()) > 0 and int(sa["decision_count"][0]) == k
            say("20,000 requests: cycle %d identical (%d blocks matched)" % (cyc, int(sa["ml"].sum())))
            now += 1000
    finally:
        api.sae_destroy(a.ctx)
        api.sae_destroy(b.ctx)


def test_batched_engine_context():
    cfg = synth.pool_config("tiny")
    pool = synth.make_pool(cfg, n_blocks=4096, seed=3)
    k = 32
    p = Pair(cfg["kinds"], pool, k, mu=cfg["mu"], sigma=cfg["sigma"], K=k)
    rng = np.random.default_rng(8)
    try:
        R, L = synth.make_requests(pool["chains"], 50, cfg["req_len"], cfg["hit_frac"], rng)
        p.match_select(R, L, pool["now"], PM, pool["now"], k, commit=True)
        p.check_counters()
        p.check_pool()
        assert not p.status()
    finally:
        p.close()


def test_argument_errors_fail_before_any_work():
    cfg = synth.pool_config("tiny")
    pool = synth.make_pool(cfg, n_blocks=20000, seed=4)
    p = Pair(cfg["kinds"], pool, 16)
    try:
        R, L = synth.make_requests(pool["chains"], 4, 8, 1.0, 1)
        hd = torch.as_tensor(u64(R).view(np.int64)).cuda()
        ld = torch.as_tensor(L).cuda()
        ml = torch.full((len(L),), -7, dtype=torch.int32, device="cuda")
        with pytest.raises(api.SaeError):
            api.sae_match_select(p.ctx, hd, ld, pool["now"], 1 << 7, ml, pool["now"], 4, 0, p.out.victims,
                                 p.out.count, p.out.decision, p.out.decision_count)
        with pytest.raises(api.SaeError):
            api.sae_match_select(p.ctx, hd, ld, pool["now"], PM, ml, pool["now"], 17, 0, p.out.victims,
                                 p.out.count, p.out.decision, p.out.decision_count)
        torch.cuda.synchronize()
        assert (ml == -7).all(), "a rejected call wrote match lengths"
    finally:
        p.close()
