"""Determinism of the HIP path (GPU).  Two contexts built from the same pools
and driven by the same calls end every cycle with the same results bit for
bit -- every list, score bit, decision entry, match length and matched id,
the counters, the learned parameters, the interval buffers and every pool
array -- although their kernels append candidates, hits and victims with
atomics in whatever order the hardware runs them.

 * Mid pool (262,144 blocks, 3 queues, k = 1,024; pool-scan engine), every
   learner on: per cycle a selection without commit overlapped by a
   read-only prefix match on a second stream, then decision + commit, a
   touching prefix match with statistics and intervals, Add() of fresh
   blocks into the freed slots, feedback.
 * 64 instances of 16,384 blocks (batched engine), k = 64: the same cycle,
   requests spread over the instances."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

import synth  # noqa: E402
from harness import say, u64  # noqa: E402
from paper_2605_18825_amd import api  # noqa: E402
from paper_2605_18825_amd.pool import DevicePool, SelectBuffers  # noqa: E402

LEARN = api.LEARN_TOKEN_WEIGHTS | api.LEARN_QUEUE_WEIGHTS | api.LEARN_LOGNORMAL | api.LEARN_DECAY_POWER
POOL_FIELDS = ("last_access", "meta", "off", "hash", "parent", "child_count", "ref_count", "access_count")
PM_ALL = api.PM_TOUCH | api.PM_STATS | api.PM_INTERVALS


class Run:
    """One context over n_inst instances, filled from `pools`."""

    def __init__(self, pools, cfg, k, max_req):
        self.n_inst, self.N = len(pools), pools[0]["n_blocks"]
        self.kinds = cfg["kinds"]
        self.Q = len(self.kinds)
        self.ctx = api.sae_create(self.n_inst, self.N, self.kinds, max_k=k, max_requests=max_req)
        self.dp = DevicePool(self.n_inst, self.N)
        for i, p in enumerate(pools):
            self.dp.fill_instance(i, p)
        self.dp.bind(self.ctx)
        api.sae_index_build(self.ctx)
        api.sae_set_params(self.ctx, -1, api.make_params(self.Q, mu=cfg["mu"], sigma=cfg["sigma"], K=k,
                                                         learn=LEARN))
        self.out = SelectBuffers(self.n_inst, self.Q, k)
        self.out2 = SelectBuffers(self.n_inst, self.Q, k)

    def close(self):
        api.sae_destroy(self.ctx)

    def snapshot(self, extra):
        """Everything the calls produced or changed, as host arrays."""
        torch.cuda.synchronize()
        snap = {f: getattr(self.dp, f).cpu().numpy().copy() for f in POOL_FIELDS}
        for name, o in (("sel", self.out), ("sel_overlapped", self.out2)):
            snap[name + ".victims"] = o.victims.cpu().numpy()
            snap[name + ".scores"] = o.scores.cpu().numpy().view(np.uint32)
            snap[name + ".count"] = o.count.cpu().numpy()
            snap[name + ".decision"] = o.decision.cpu().numpy()
            snap[name + ".decision_count"] = o.decision_count.cpu().numpy()
        for i in range(self.n_inst):
            c = api.sae_get_counters(self.ctx, i)
            p = api.sae_get_params(self.ctx, i)
            snap["counters%d" % i] = np.array(list(c.evicted) + list(c.missed) + list(c.hits) + list(c.evictions) +
                                             list(c.bin_hits) + list(c.bin_missed) + list(c.type_hits) +
                                             list(c.type_added) + list(c.resident) +
                                             [c.eviction_count, c.pending, c.n_updates], np.int64)
            snap["params%d" % i] = np.array(list(p.w) + list(p.alpha) + list(p.mu) + list(p.sigma) + [p.gamma],
                                           np.float32).view(np.uint32)
            for q in range(self.Q):
                if self.kinds[q] == api.KIND_LOGNORMAL:
                    snap["ivl%d.%d" % (i, q)] = np.array(api.sae_get_intervals(self.ctx, i, q), np.int32)
        for key, t in extra.items():
            snap[key] = t.cpu().numpy().copy()
        snap["status"] = np.array(api.status_names(api.sae_poll_status(self.ctx)), dtype=object)
        return snap


def cycle_inputs(rng, pools, cfg, n_req, req_len, k, now):
    """One cycle's requests (hashes, lengths, instances) and Add() arrays."""
    n_inst = len(pools)
    R, L = synth.make_requests(pools[0]["chains"], n_req, req_len, cfg["hit_frac"], rng)
    inst = rng.integers(0, n_inst, n_req).astype(np.int32)
    for j in range(n_req):  # a hit request follows a chain of its own instance
        if inst[j]:
            R2, _ = synth.make_requests(pools[inst[j]]["chains"], 1, req_len, cfg["hit_frac"], rng)
            R[j, :L[j]] = R2[0, :L[j]]
    hashes = synth.pools._fix_reserved(rng.integers(1, 2 ** 63, (n_inst, k), dtype=np.uint64))
    queue = rng.choice(len(cfg["kinds"]), size=(n_inst, k), p=cfg["mix"]).astype(np.int32)
    counts = synth.pools.token_type_counts(rng, n_inst * k).reshape(n_inst, k, 5)
    omax = rng.integers(31, 251, (n_inst, k)).astype(np.int32)
    ob = (rng.random((n_inst, k)) * (omax + 1)).astype(np.int32).clip(0, omax)
    return R, L, inst, hashes, queue, counts, omax, ob


def drive(run, inp, now, k, streams):
    """One cycle on one context; the device tensors it wrote are returned."""
    R, L, inst, hashes, queue, counts, omax, ob = inp
    sa, sb = streams
    n_inst, n = run.n_inst, len(L)
    dev = lambda a, dt: torch.as_tensor(np.ascontiguousarray(a)).to(device="cuda", dtype=dt)
    hd, ld, idev = dev(u64(R).view(np.int64), torch.int64), dev(L, torch.int32), dev(inst, torch.int32)
    ml_ro = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    mid_ro = torch.full(hd.shape, -7, dtype=torch.int32, device="cuda")
    ml = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    mid = torch.full(hd.shape, -7, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    # a selection without commit overlapped by a read-only prefix match
    run.out2.run(run.ctx, now, k, 0, stream=sa)
    api.sae_prefix_match(run.ctx, hd, ld, now, 0, ml_ro, matched_ids=mid_ro, inst=idev, stream=sb)
    torch.cuda.synchronize()
    # the serving cycle
    run.out.run(run.ctx, now, k, api.SS_COMMIT)
    api.sae_prefix_match(run.ctx, hd, ld, now + 1, PM_ALL, ml, matched_ids=mid, inst=idev)
    d = run.out.decision_count.cpu().numpy()
    dec = run.out.decision.cpu().numpy()
    ids = np.concatenate([dec[i, :d[i]] for i in range(n_inst)]).astype(np.int32)
    iv = np.concatenate([np.full(d[i], i, np.int32) for i in range(n_inst)])
    pos = np.concatenate([np.arange(d[i]) for i in range(n_inst)])
    if len(ids):
        tau = torch.empty(len(ids), dtype=torch.uint8, device="cuda")
        api.sae_block_type(dev(counts[iv, pos], torch.uint8).reshape(len(ids), 5).contiguous(), tau)
        meta = api.meta_to_u16(api.pack_meta(dev(queue[iv, pos], torch.int32), tau.to(torch.int32),
                                             dev(np.full(len(ids), 16), torch.int32)))
        off = api.off_to_u32(api.pack_off(dev(ob[iv, pos], torch.int64), dev(omax[iv, pos], torch.int64)))
        api.sae_insert_blocks(run.ctx, dev(ids, torch.int32), dev(u64(hashes[iv, pos]).view(np.int64), torch.int64),
                              dev(np.full(len(ids), -1), torch.int32), dev(np.full(len(ids), now + 2), torch.int32),
                              meta, off, inst=dev(iv, torch.int32))
    api.sae_feedback_update(run.ctx, 0)
    return {"ml_ro": ml_ro, "mid_ro": mid_ro, "ml": ml, "mid": mid}


def compare(a, b, cyc):
    assert a.keys() == b.keys()
    for key in a:
        if a[key].dtype == object:
            assert list(a[key]) == list(b[key]), "cycle %d: %s differs" % (cyc, key)
            continue
        if not np.array_equal(a[key], b[key]):
            bad = np.argwhere(a[key] != b[key])[:5].tolist()
            raise AssertionError("cycle %d: %s differs at %s" % (cyc, key, bad))


def run_pair(pools, cfg, k, n_req, req_len, cycles, seed, label):
    max_req = n_req
    a, b = Run(pools, cfg, k, max_req), Run(pools, cfg, k, max_req)
    streams = (torch.cuda.Stream(), torch.cuda.Stream())
    rng = np.random.default_rng(seed)
    now = max(p["now"] for p in pools)
    try:
        for cyc in range(cycles):
            inp = cycle_inputs(rng, pools, cfg, n_req, req_len, k, now)
            sa = a.snapshot(drive(a, inp, now, k, streams))
            sb = b.snapshot(drive(b, inp, now, k, streams))
            compare(sa, sb, cyc)
            say("%s: cycle %d identical (%d victims, %d matched)" % (label, cyc, int(sa["sel.decision_count"].sum()),
                                                                      int(sa["ml"].sum())))
            now += 1000
        assert sum(int(x) for x in sa["sel.decision_count"]) > 0 and int(sa["ml"].sum()) > 0
    finally:
        a.close()
        b.close()


def test_mid_pool_runs_are_identical():
    cfg = synth.pool_config("mid")
    pool = synth.make_pool(cfg)
    run_pair([pool], cfg, cfg["k"], cfg["n_req"], cfg["req_len"], 6, cfg["seed"] + 21, "determinism mid")


def test_batched_instances_runs_are_identical():
    cfg = synth.pool_config("tiny")
    pools = [synth.make_pool(cfg, n_blocks=16384, seed=500 + i) for i in range(64)]
    run_pair(pools, cfg, cfg["k"], 1024, cfg["req_len"], 6, 77, "determinism batched")
