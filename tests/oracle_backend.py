"""The oracle as a trace-replay backend: one OracleCache per replayed instance,
the same interface as paper_2605_18825_amd.engine.DeviceBackend."""
import numpy as np

import oracle


class OracleBackend:
    def __init__(self, insts, capacity, kinds, roles, mu, sigma, K, learn, w=1.0, alpha=1.0, gamma=1.0, eta=0.01,
                 T=1.0, beta=0.1, ghost_window=None, cascade=False):
        self.insts = list(insts)
        self.intervals = bool(learn & 4)
        self.cascade = bool(cascade)  # Algorithm 1 one victim at a time instead of a snapshot decision
        self.roles = list(roles)
        self.Q = len(kinds)
        self.c = {}
        for i in self.insts:
            prm = oracle.Params(self.Q, w=w, alpha=alpha, mu=mu, sigma=sigma, gamma=gamma, eta=eta, T=T, beta=beta,
                                K=K, learn_w=bool(learn & 1), learn_alpha=bool(learn & 2), learn_ln=bool(learn & 4),
                                learn_gamma=bool(learn & 8), learn_w_ema=bool(learn & 16),
                                learn_alpha_rel=bool(learn & 32))
            self.c[i] = oracle.OracleCache(capacity, kinds, prm, ghost_window=ghost_window)

    def prefix_match(self, now, insts, prompts):
        ml = np.zeros(len(insts), np.int32)
        mids = []
        for j, (i, p) in enumerate(zip(insts, prompts)):
            m, ids = self.c[i].prefix_match(np.asarray(p, np.uint64)[None, :], [len(p)], now, touch=True, stats=True,
                                            intervals=self.intervals)
            ml[j] = m[0]
            mids.append(ids[0, :m[0]].astype(np.int32))
        return ml, mids

    def ref(self, inst, ids, delta):
        for i in self.insts:
            sel = inst == i
            if sel.any():
                self.c[i].ref(ids[sel], delta)

    def evict(self, now, k):
        out = {}
        for i in self.insts:
            if k[i] > 0 and self.cascade:
                dec = self.c[i].decide_cascade(now, int(k[i]))
                self.c[i].commit(dec)
                out[i] = dec
            elif k[i] > 0:
                _, _, dec = self.c[i].score_select(now, int(k[i]), commit=True)
                out[i] = dec
            else:
                out[i] = np.zeros(0, np.int32)
        return out

    def insert(self, now, f):
        counts = np.zeros((len(f["ids"]), 5), np.uint8)
        counts[np.arange(len(f["ids"])), f["types"]] = 16
        tau = oracle.block_type(counts)
        queue = oracle.classify(tau, f["hints"], self.roles)
        for i in self.insts:
            sel = f["inst"] == i
            if not sel.any():
                continue
            n = int(sel.sum())
            self.c[i].insert(f["ids"][sel], f["hash"][sel], f["parent"][sel], np.full(n, now, np.int32),
                             queue[sel], tau[sel], np.full(n, 16, np.int32), f["ob"][sel], f["omax"][sel])

    def feedback(self):
        for i in self.insts:
            self.c[i].feedback()

    def counters(self, i):
        d = self.c[i].counters()
        d["n_updates"] = self.c[i].n_updates
        return d

    def params(self, i):
        p = self.c[i].prm
        return p.w.copy(), p.alpha.copy()

    def timing_params(self, i):
        p = self.c[i].prm
        return p.mu.copy(), p.sigma.copy(), np.float32(p.gamma)
