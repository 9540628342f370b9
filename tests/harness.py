"""Side-by-side runner: the CPU oracle and the HIP path on identical inputs.

Used by the GPU parity tests only.  Inputs come from synth (seeded); the oracle
never sees a value produced by the HIP path, and vice versa.
"""
import sys

import numpy as np
import torch

import oracle
from paper_2605_18825_amd import api
from paper_2605_18825_amd.pool import DevicePool, SelectBuffers


_capman = None  # pytest's capture manager, set by conftest: progress lines bypass output capture


def set_capture_manager(capman):
    global _capman
    _capman = capman


def say(*a):
    """A progress line, shown as the test runs even when pytest captures
    output (a long GPU test then keeps printing)."""
    if _capman is not None:
        with _capman.global_and_fixture_disabled():
            print(*a, flush=True)
    else:
        print(*a, flush=True)
        sys.stdout.flush()


def u64(a):
    return np.asarray(a, np.uint64)


def gpu_insert(ctx, ids, hashes, parent, la, queue, counts, ntok, ob, omax):
    """Add() of host arrays on the HIP side; block types from the token counts
    by sae_block_type."""
    n = len(ids)
    if n == 0:
        return
    counts = np.asarray(counts, np.uint8)
    dev = lambda a, dt: torch.as_tensor(np.ascontiguousarray(a)).to(device="cuda", dtype=dt)
    tau = torch.empty(n, dtype=torch.uint8, device="cuda")
    api.sae_block_type(dev(counts, torch.uint8).reshape(n, 5).contiguous(), tau)
    meta = api.meta_to_u16(api.pack_meta(dev(queue, torch.int32), tau.to(torch.int32), dev(ntok, torch.int32)))
    off = api.off_to_u32(api.pack_off(dev(ob, torch.int64), dev(omax, torch.int64)))
    api.sae_insert_blocks(ctx, dev(ids, torch.int32), dev(u64(hashes).view(np.int64), torch.int64),
                          dev(parent, torch.int32), dev(la, torch.int32), meta, off)


class Pair:
    """One instance held by both the oracle and a libsae context."""

    def __init__(self, kinds, pool, max_k, mu=None, sigma=None, gamma=1.0, w=1.0, alpha=1.0, K=None,
                 ghost_window=0, learn=3, eta=0.01, T=1.0, beta=0.1, beta_ln=0.1, max_requests=0):
        N = pool["n_blocks"]
        Q = len(kinds)
        self.N, self.Q, self.max_k, self.kinds = N, Q, max_k, list(kinds)
        mu = [0.0] * Q if mu is None else list(mu)
        sigma = [1.0] * Q if sigma is None else list(sigma)
        K = max_k if K is None else K
        self.prm = oracle.Params(Q, w=w, alpha=alpha, mu=mu, sigma=sigma, gamma=gamma, eta=eta, T=T, beta=beta, K=K,
                                 learn_w=bool(learn & 1), learn_alpha=bool(learn & 2), beta_ln=beta_ln,
                                 learn_ln=bool(learn & 4), learn_gamma=bool(learn & 8),
                                 learn_w_ema=bool(learn & 16), learn_alpha_rel=bool(learn & 32))
        self.oc = oracle.OracleCache(N, kinds, self.prm, ghost_window=ghost_window or None)
        self.tau_oracle = oracle.block_type(pool["counts"])
        self.oc.bind(pool["last_access"], pool["queue"], self.tau_oracle, pool["ntok"], pool["ob"], pool["omax"],
                     pool["valid"], pool["ref_count"], pool["parent"], pool["hash"], pool.get("access_count"))
        self.ctx = api.sae_create(1, N, kinds, max_k=max_k, ghost_window=ghost_window, max_requests=max_requests)
        self.dp = DevicePool(1, N)
        self.tau_gpu = self.dp.fill_instance(0, pool)
        self.dp.bind(self.ctx)
        api.sae_index_build(self.ctx)
        wv = list(w) if hasattr(w, "__len__") else w
        av = list(alpha) if hasattr(alpha, "__len__") else alpha
        api.sae_set_params(self.ctx, -1, api.make_params(Q, w=wv, alpha=av, mu=mu, sigma=sigma, gamma=gamma, eta=eta,
                                                         temperature=T, beta=beta, K=K, learn=learn,
                                                         beta_ln=beta_ln))
        self.out = SelectBuffers(1, Q, max_k)

    def close(self):
        api.sae_destroy(self.ctx)

    # ------------------------------------------------------------ comparisons
    def check_tau(self):
        g = self.tau_gpu.cpu().numpy().astype(np.int32)
        assert np.array_equal(g, self.tau_oracle), "block types differ at %s" % np.nonzero(g != self.tau_oracle)[0][:10]

    def select(self, now, k, flags=0, commit=False, check=True):
        """Run both sides; compare per-queue victims, their key bits and the
        decision element by element.  With api.SS_CASCADE the oracle's decision
        is its sequential cascade (the per-queue lists stay the snapshot's)."""
        if commit:
            flags |= api.SS_COMMIT
        self.out.run(self.ctx, now, k, flags)
        lists, key, dec = self._oracle_select(now, k, flags)
        if check:
            self._check_select(lists, key, dec)
        return lists, key, dec

    def _oracle_select(self, now, k, flags):
        commit = bool(flags & api.SS_COMMIT)
        if flags & api.SS_CASCADE:
            lists, key, _ = self.oc.select_per_queue(now, k)
            dec = self.oc.decide_cascade(now, k)
            if commit:
                self.oc.commit(dec)
            return lists, key, dec
        return self.oc.score_select(now, k, commit=commit)

    def _check_select(self, lists, key, dec):
        torch.cuda.synchronize()
        cnt = self.out.count[0].cpu().numpy()
        vic = self.out.victims[0].cpu().numpy()
        sc = self.out.scores[0].cpu().numpy().view(np.uint32)
        for q in range(self.Q):
            c = int(cnt[q])
            want = lists[q]
            assert c == len(want), "queue %d: count %d vs oracle %d" % (q, c, len(want))
            got = vic[q, :c]
            if not np.array_equal(got, want):
                bad = np.nonzero(got != want)[0][0]
                raise AssertionError("queue %d: first difference at position %d: gpu %d (key %08x) vs oracle %d "
                                     "(key %08x)" % (q, bad, got[bad], sc[q, bad], want[bad], key[want[bad]]))
            assert np.array_equal(sc[q, :c], key[want]), "queue %d: score bits differ" % q
        d = int(self.out.decision_count[0])
        assert d == len(dec), "decision size %d vs %d" % (d, len(dec))
        assert np.array_equal(self.out.decision[0, :d].cpu().numpy(), dec), "decision differs"

    def _pm_buffers(self, hashes, lens):
        R = torch.as_tensor(u64(hashes).view(np.int64)).cuda()
        L = torch.as_tensor(np.asarray(lens, np.int32)).cuda()
        ml = torch.zeros(len(lens), dtype=torch.int32, device="cuda")
        mid = torch.zeros(R.shape, dtype=torch.int32, device="cuda")
        return R, L, ml, mid

    def _oracle_pm(self, hashes, lens, now, flags):
        return self.oc.prefix_match(hashes, lens, now, touch=bool(flags & api.PM_TOUCH),
                                    stats=bool(flags & api.PM_STATS), intervals=bool(flags & api.PM_INTERVALS))

    @staticmethod
    def _check_pm(ml, mid, om, omid):
        torch.cuda.synchronize()
        g = ml.cpu().numpy()
        assert np.array_equal(g, om), "match_len differs at %s" % np.nonzero(g != om)[0][:10]
        assert np.array_equal(mid.cpu().numpy(), omid), "matched ids differ"

    def prefix_match(self, hashes, lens, now, flags, check=True):
        R, L, ml, mid = self._pm_buffers(hashes, lens)
        api.sae_prefix_match(self.ctx, R, L, now, flags, ml, matched_ids=mid)
        om, omid = self._oracle_pm(hashes, lens, now, flags)
        if check:
            self._check_pm(ml, mid, om, omid)
        return om

    def match_select(self, hashes, lens, pm_now, pm_flags, now, k, flags=0, commit=False):
        """sae_match_select on the GPU; on the oracle its prefix match and then
        its selection.  Both halves are compared as prefix_match() and
        select() compare them."""
        if commit:
            flags |= api.SS_COMMIT
        R, L, ml, mid = self._pm_buffers(hashes, lens)
        self.out.run_after_match(self.ctx, R, L, pm_now, pm_flags, ml, now, k, flags, matched_ids=mid)
        om, omid = self._oracle_pm(hashes, lens, pm_now, pm_flags)
        lists, key, dec = self._oracle_select(now, k, flags)
        self._check_pm(ml, mid, om, omid)
        self._check_select(lists, key, dec)
        return om, dec

    def insert(self, ids, hashes, parent, la, queue, counts_or_tau, ntok, ob, omax, tau_given=None):
        """Add() on both sides.  Block types: the oracle computes its own from
        the token counts; the HIP side from the same counts via sae_block_type."""
        counts = np.asarray(counts_or_tau, np.uint8)
        tau_o = oracle.block_type(counts)
        self.oc.insert(ids, hashes, parent, la, queue, tau_o, ntok, ob, omax)
        gpu_insert(self.ctx, ids, hashes, parent, la, queue, counts, ntok, ob, omax)

    def feedback(self, force=False):
        api.sae_feedback_update(self.ctx, api.FB_FORCE if force else 0)
        return self.oc.feedback(force=force)

    def check_params(self):
        gp = api.sae_get_params(self.ctx, 0)
        gw = np.array(gp.w[:5], np.float32)
        ga = np.array(gp.alpha[:self.Q], np.float32)
        assert np.array_equal(gw.view(np.uint32), self.prm.w.view(np.uint32)), "w: %s vs %s" % (gw, self.prm.w)
        assert np.array_equal(ga.view(np.uint32), self.prm.alpha.view(np.uint32)), "alpha: %s vs %s" % (ga, self.prm.alpha)
        gm = np.array(gp.mu[:self.Q], np.float32)
        gs = np.array(gp.sigma[:self.Q], np.float32)
        assert np.array_equal(gm.view(np.uint32), self.prm.mu.view(np.uint32)), "mu: %s vs %s" % (gm, self.prm.mu)
        assert np.array_equal(gs.view(np.uint32), self.prm.sigma.view(np.uint32)), \
            "sigma: %s vs %s" % (gs, self.prm.sigma)
        gg = np.float32(gp.gamma)
        assert gg.view(np.uint32) == np.float32(self.prm.gamma).view(np.uint32), \
            "gamma: %r vs %r" % (gg, self.prm.gamma)

    def check_intervals(self):
        for q in range(self.Q):
            if self.kinds[q] == api.KIND_LOGNORMAL:
                got = api.sae_get_intervals(self.ctx, 0, q)
                want = self.oc.ivl[q]
                assert got == want, "queue %d intervals: %d held vs oracle %d; first %s vs %s" % (
                    q, len(got), len(want), got[:5], want[:5])

    def check_counters(self):
        c = api.sae_get_counters(self.ctx, 0)
        o = self.oc
        assert list(c.evicted) == o.evicted, ("evicted", list(c.evicted), o.evicted)
        assert list(c.missed) == o.missed, ("missed", list(c.missed), o.missed)
        assert list(c.hits[:self.Q]) == o.hits, ("hits", list(c.hits[:self.Q]), o.hits)
        assert list(c.evictions[:self.Q]) == o.evictions, ("evictions", list(c.evictions[:self.Q]), o.evictions)
        assert c.eviction_count == o.ev_count
        assert bool(c.pending) == o.pending
        assert list(c.bin_hits) == o.bin_hits, ("bin_hits", list(c.bin_hits), o.bin_hits)
        assert list(c.bin_missed) == o.bin_missed, ("bin_missed", list(c.bin_missed), o.bin_missed)
        assert list(c.type_hits) == o.type_hits, ("type_hits", list(c.type_hits), o.type_hits)
        assert list(c.type_added) == o.type_added, ("type_added", list(c.type_added), o.type_added)
        assert list(c.resident[:self.Q]) == o.resident(), ("resident", list(c.resident[:self.Q]), o.resident())

    def check_pool(self):
        torch.cuda.synchronize()
        m = api.unpack_meta(self.dp.meta)
        o = self.oc
        valid = m["valid"].cpu().numpy()
        assert np.array_equal(valid, o.valid), "valid bits differ"
        v = o.valid
        assert np.array_equal(m["leaf"].cpu().numpy()[v], (o.child_count == 0)[v]), "leaf bits differ"
        assert np.array_equal(m["ref"].cpu().numpy()[v], (o.ref_count > 0)[v]), "ref bits differ"
        assert np.array_equal(self.dp.child_count.cpu().numpy()[v], o.child_count[v]), "child counts differ"
        assert np.array_equal(self.dp.last_access.cpu().numpy()[v], o.la[v]), "last_access differs"
        assert np.array_equal(self.dp.access_count.cpu().numpy()[v], o.access_count[v]), "access_count differs"

    def status(self):
        return api.status_names(api.sae_poll_status(self.ctx))
