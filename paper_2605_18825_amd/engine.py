"""A batched block-manager adapter over libsae for trace replay.

One context holds n_inst independent caches.  Each method marshals one
batched C-ABI call (all instances at once) and copies back what the caller's
block manager needs on the host: match lengths and matched block ids, and
eviction decisions.  No policy step runs here.

Host arrays go to the device through pinned staging buffers with
asynchronous copies, and results come back the same way with one stream
synchronisation per call that returns them, so a replay step costs few
host-device round trips.  Everything runs on the stream that was current when
the backend was made (library calls name it; torch's copies use the current
stream), so the caller keeps that stream current.
"""
import numpy as np
import torch

from . import api
from .pool import DevicePool, SelectBuffers


class _Staging:
    """Pinned host buffers and device buffers, reused call after call, on one
    stream.

    put(name, array) copies a host array into the pinned buffer `name` and
    from there, asynchronously on the stream, into the device buffer `name`;
    it returns the device view.  Before a pinned input buffer is written
    again, the copy that last read it must have finished (its event); the
    device buffer needs no such wait, since everything runs on one stream.
    get(name, t) starts the copy of t into a pinned output buffer; its caller
    synchronises the stream before reading it and before the next get."""

    def __init__(self, stream):
        self.stream = stream
        self.host = {}
        self.dev = {}
        self.ev = {}

    def _bufs(self, name, nbytes, device=True):
        h = self.host.get(name)
        if h is None or h.numel() < nbytes:
            n = max(nbytes, 2 * (h.numel() if h is not None else 0), 4096)
            if name in self.ev:
                self.ev[name].synchronize()
            self.host[name] = torch.empty(n, dtype=torch.uint8, pin_memory=True)
            if device:
                self.dev[name] = torch.empty(n, dtype=torch.uint8, device="cuda")
                self.ev[name] = torch.cuda.Event()
                self.ev[name].record(self.stream)
        return self.host[name], self.dev.get(name)

    def put(self, name, a, dtype):
        a = np.ascontiguousarray(a)
        nb = a.nbytes
        h, d = self._bufs(name, max(nb, 1))
        self.ev[name].synchronize()
        h.numpy()[:nb] = a.view(np.uint8).ravel()
        d[:nb].copy_(h[:nb], non_blocking=True)
        self.ev[name].record(self.stream)
        return d[:nb].view(dtype).view(a.shape) if nb else d[:0].view(dtype)

    def get(self, name, t):
        """Start copying device tensor t into the pinned buffer `name`; the
        numpy view is valid after the stream has been synchronised."""
        t = t.contiguous()
        nb = t.numel() * t.element_size()
        h, _ = self._bufs("out_" + name, max(nb, 1), device=False)
        h[:nb].copy_(t.view(-1).view(torch.uint8), non_blocking=True)
        return h[:nb].numpy()


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
        self.stream = torch.cuda.current_stream()
        self.st = _Staging(self.stream)
        self.select_calls = 0

    def close(self):
        self.stream.synchronize()
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
        hd = self.st.put("pm_h", h.view(np.int64), torch.int64)
        ld = self.st.put("pm_len", lens, torch.int32)
        idv = self.st.put("pm_inst", np.asarray(insts, np.int32), torch.int32)
        ml = torch.empty(n, dtype=torch.int32, device="cuda")
        mid = torch.empty((n, L), dtype=torch.int32, device="cuda")
        flags = api.PM_TOUCH | api.PM_STATS | (api.PM_INTERVALS if self.intervals else 0)
        api.sae_prefix_match(self.ctx, hd, ld, now, flags, ml, matched_ids=mid, inst=idv, stream=self.stream)
        mlh = self.st.get("pm_ml", ml)
        midh = self.st.get("pm_mid", mid)
        self.stream.synchronize()
        mlv = mlh.view(np.int32)[:n].copy()
        midv = midh.view(np.int32)[:n * L].reshape(n, L)
        return mlv, [midv[j, :mlv[j]].copy() for j in range(n)]

    def ref(self, inst, ids, delta):
        if len(ids):
            both = np.stack([np.asarray(inst, np.int32), np.asarray(ids, np.int32)])
            d = self.st.put("ref%d" % (delta > 0), both, torch.int32)
            api.sae_ref_blocks(self.ctx, d[1], delta, inst=d[0], stream=self.stream)

    def evict(self, now, k):
        k = np.asarray(k, np.int32)
        if self.n_inst == 1:  # one cache: k goes by value
            self.out.run(self.ctx, now, int(k[0]), self.select_flags, stream=self.stream)
        else:
            kd = self.st.put("k", k, torch.int32)
            self.out.run(self.ctx, now, self.max_k, self.select_flags, k_per_inst=kd, stream=self.stream)
        self.select_calls += 1
        small = self.n_inst * self.max_k <= 16384
        cnt = self.st.get("cnt", self.out.decision_count)
        if small:  # the whole decision buffer comes back with the counts
            dec = self.st.get("dec", self.out.decision)
        self.stream.synchronize()
        cnt = cnt.view(np.int32)[:self.n_inst].copy()
        m = int(cnt.max()) if len(cnt) else 0
        if m == 0:
            return [np.zeros(0, np.int32) for _ in range(self.n_inst)]
        if small:
            dec = dec.view(np.int32)[:self.n_inst * self.max_k].reshape(self.n_inst, self.max_k)
        else:
            dec = self.st.get("dec", self.out.decision[:, :m])
            self.stream.synchronize()
            dec = dec.view(np.int32)[:self.n_inst * m].reshape(self.n_inst, m)
        return [dec[i, :cnt[i]].copy() for i in range(self.n_inst)]

    def insert(self, now, f):
        n = len(f["ids"])
        types = np.asarray(f["types"])
        # int32 columns: instance, id, parent, last_access, off (o_b | o_max << 16 as 32-bit pattern)
        off = (np.asarray(f["omax"], np.int64) << 16) | (np.asarray(f["ob"], np.int64) & 0xFFFF)
        cols = np.stack([np.asarray(f["inst"], np.int32), np.asarray(f["ids"], np.int32),
                         np.asarray(f["parent"], np.int32), np.full(n, now, np.int32),
                         off.astype(np.uint32).view(np.int32)])
        # uint8 columns: token-type counts of one-type blocks (16 tokens of the block's type), hints
        u8 = np.zeros((n, 6), np.uint8)
        u8[np.arange(n), types] = 16
        u8[:, 5] = f["hints"]
        ci = self.st.put("ins_i32", cols, torch.int32)
        cb = self.st.put("ins_u8", u8, torch.uint8)
        hd = self.st.put("ins_h", np.asarray(f["hash"], np.uint64).view(np.int64), torch.int64)
        counts = cb[:, :5].contiguous()
        hints = cb[:, 5].contiguous()
        tau = torch.empty(n, dtype=torch.uint8, device="cuda")
        api.sae_block_type(counts, tau, stream=self.stream)
        # meta before Classify: type, num_tokens - 1 = 15 (the queue bits are Classify's)
        meta = ((tau.to(torch.int32) << 3) | (15 << 9)).to(torch.int16)
        api.sae_classify_blocks(self.ctx, hints, meta, self.roles, stream=self.stream)
        api.sae_insert_blocks(self.ctx, ci[1], hd, ci[2], ci[3], meta, ci[4], inst=ci[0], stream=self.stream)

    def feedback(self):
        api.sae_feedback_update(self.ctx, 0, stream=self.stream)

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
