"""A batched block-manager adapter over libsae for trace replay.

One context holds n_inst independent caches.  Each method marshals one
batched C-ABI call (all instances at once) and copies back what the caller's
block manager needs on the host: match lengths and matched block ids, and
eviction decisions.  No policy step runs here.
"""
import numpy as np
import torch

from . import api
from .pool import DevicePool, SelectBuffers


def _dev(a, dtype):
    return torch.as_tensor(np.ascontiguousarray(a)).to(device="cuda", dtype=dtype)


class DeviceBackend:
    def __init__(self, n_inst, capacity, kinds, roles, max_k, mu, sigma, K, learn, w=1.0, alpha=1.0, gamma=1.0,
                 eta=0.01, T=1.0, beta=0.1, ghost_window=0, cascade=False):
        self.n_inst, self.N, self.Q = n_inst, capacity, len(kinds)
        self.roles = list(roles)
        self.max_k = max_k
        self.intervals = bool(learn & api.LEARN_LOGNORMAL)
        self.select_flags = api.SS_COMMIT | (api.SS_CASCADE if cascade else 0)
        self.ctx = api.sae_create(n_inst, capacity, kinds, max_k=max_k, ghost_window=ghost_window,
                                  max_requests=n_inst if self.intervals else 0)
        self.pool = DevicePool(n_inst, capacity)
        self.pool.bind(self.ctx)
        api.sae_index_build(self.ctx)
        api.sae_set_params(self.ctx, -1, api.make_params(self.Q, w=w, alpha=alpha, mu=mu, sigma=sigma, gamma=gamma,
                                                         eta=eta, temperature=T, beta=beta, K=K, learn=learn))
        self.out = SelectBuffers(n_inst, self.Q, max_k)
        self.select_ms = 0.0
        self.select_calls = 0

    def close(self):
        api.sae_destroy(self.ctx)

    # ---------------------------------------------------------------- calls
    def prefix_match(self, now, insts, prompts):
        n = len(prompts)
        L = max(1, max(len(p) for p in prompts))
        h = np.zeros((n, L), np.uint64)
        lens = np.zeros(n, np.int32)
        for j, p in enumerate(prompts):
            h[j, :len(p)] = p
            lens[j] = len(p)
        ml = torch.zeros(n, dtype=torch.int32, device="cuda")
        mid = torch.empty((n, L), dtype=torch.int32, device="cuda")
        flags = api.PM_TOUCH | api.PM_STATS | (api.PM_INTERVALS if self.intervals else 0)
        api.sae_prefix_match(self.ctx, _dev(h.view(np.int64), torch.int64), _dev(lens, torch.int32), now,
                             flags, ml, matched_ids=mid, inst=_dev(insts, torch.int32))
        ml = ml.cpu().numpy()
        mid = mid.cpu().numpy()
        return ml, [mid[j, :ml[j]] for j in range(n)]

    def ref(self, inst, ids, delta):
        if len(ids):
            api.sae_ref_blocks(self.ctx, _dev(ids, torch.int32), delta, inst=_dev(inst, torch.int32))

    def evict(self, now, k):
        kd = _dev(k, torch.int32)
        self.out.run(self.ctx, now, self.max_k, self.select_flags, k_per_inst=kd)
        cnt = self.out.decision_count.cpu().numpy()
        dec = self.out.decision.cpu().numpy()
        self.select_calls += 1
        return [dec[i, :cnt[i]].copy() for i in range(self.n_inst)]

    def insert(self, now, f):
        n = len(f["ids"])
        types = f["types"]
        counts = np.zeros((n, 5), np.uint8)
        counts[np.arange(n), types] = 16
        tau = torch.empty(n, dtype=torch.uint8, device="cuda")
        api.sae_block_type(_dev(counts, torch.uint8), tau)
        zeros = torch.zeros(n, dtype=torch.int32, device="cuda")
        meta = api.meta_to_u16(api.pack_meta(zeros, tau.to(torch.int32), zeros + 16))
        api.sae_classify_blocks(self.ctx, _dev(f["hints"], torch.uint8), meta, self.roles)
        off = api.off_to_u32(api.pack_off(_dev(f["ob"], torch.int64), _dev(f["omax"], torch.int64)))
        api.sae_insert_blocks(self.ctx, _dev(f["ids"], torch.int32), _dev(f["hash"].view(np.int64), torch.int64),
                              _dev(f["parent"], torch.int32), _dev(np.full(n, now, np.int32), torch.int32), meta,
                              off, inst=_dev(f["inst"], torch.int32))

    def feedback(self):
        api.sae_feedback_update(self.ctx, 0)

    # -------------------------------------------------------------- read-back
    def counters(self, i):
        c = api.sae_get_counters(self.ctx, i)
        return dict(evicted=list(c.evicted), missed=list(c.missed), hits=list(c.hits[:self.Q]),
                    evictions=list(c.evictions[:self.Q]), ev_count=int(c.eviction_count), pending=bool(c.pending),
                    n_updates=int(c.n_updates), bin_hits=list(c.bin_hits), bin_missed=list(c.bin_missed),
                    type_hits=list(c.type_hits), type_added=list(c.type_added), resident=list(c.resident[:self.Q]))

    def params(self, i):
        p = api.sae_get_params(self.ctx, i)
        return np.array(p.w[:5], np.float32), np.array(p.alpha[:self.Q], np.float32)

    def timing_params(self, i):
        """mu, sigma per queue and gamma of instance i."""
        p = api.sae_get_params(self.ctx, i)
        return np.array(p.mu[:self.Q], np.float32), np.array(p.sigma[:self.Q], np.float32), np.float32(p.gamma)

    def status(self):
        return api.status_names(api.sae_poll_status(self.ctx))
