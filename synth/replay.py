"""Trace replay: a serving engine's block manager around an eviction policy.

The replay is policy-agnostic.  It hands every backend the same requests and
uses only what the backend returns (match lengths, matched block ids,
eviction decisions), so two backends that agree produce the same run.  It
holds none of the eviction method's arithmetic.

Per request (one request per cache instance per step, all instances at the
same time `now`; the paper injects requests at a fixed interval):

1. requests that started `concurrency` or more requests earlier on the same
   instance have finished: their blocks are released (reference count - 1);
2. strict prefix matching of the prompt's block hashes (touching the hits and
   counting queue hits);
3. the matched blocks are referenced;
4. need = blocks of the sequence (prompt + generated) after the match.  While
   an instance has fewer free slots than it needs, it asks for an eviction
   decision of k = clip(need - free, k_min, max_k) victims (a decision may
   return fewer; a decision that frees nothing ends the cascade).  Victims go
   to the instance's free-slot stack;
5. the blocks after the match are inserted (Algorithm 1 Add, routed by
   Classify from their hints) into free slots, as many as there are slots,
   each a child of the block before it; o_b is the block's position and
   o_max the request's last position;
6. the inserted blocks are referenced; the learners run if due.
"""
from collections import deque

import numpy as np


class Replay:
    def __init__(self, backend, n_inst, capacity, k_min=1, max_k=1024, concurrency=4, insts=None):
        self.be = backend
        self.n_inst = n_inst
        self.capacity = capacity
        self.k_min = k_min
        self.max_k = max_k
        self.concurrency = concurrency
        self.insts = list(range(n_inst)) if insts is None else list(insts)
        self.free = {i: list(range(capacity - 1, -1, -1)) for i in self.insts}
        self.inflight = {i: deque() for i in self.insts}
        # per instance: requests, prompt blocks, hit blocks, inserted, evicted, decisions, not cached
        self.stats = {i: np.zeros(7, np.int64) for i in self.insts}

    def step(self, reqs):
        """reqs: {instance: request} for instances of this replay.  Returns
        {instance: (match_len, [decision arrays])}."""
        insts = [i for i in self.insts if i in reqs]
        if not insts:
            return {}
        now = reqs[insts[0]]["now"]
        assert all(reqs[i]["now"] == now for i in insts)
        # 1. release finished requests
        rel_i, rel_b = [], []
        for i in insts:
            dq = self.inflight[i]
            while len(dq) >= self.concurrency:
                ids = dq.popleft()
                rel_i.append(np.full(len(ids), i, np.int32))
                rel_b.append(ids)
        if rel_b:
            self.be.ref(np.concatenate(rel_i), np.concatenate(rel_b), -1)
        # 2. prefix match
        ml, mids = self.be.prefix_match(now, insts, [reqs[i]["hashes"][:reqs[i]["n_prompt"]] for i in insts])
        # 3. reference the hits
        hit_i = [np.full(len(m), i, np.int32) for i, m in zip(insts, mids)]
        if sum(len(m) for m in mids):
            self.be.ref(np.concatenate(hit_i), np.concatenate(mids).astype(np.int32), +1)
        need = {}
        for j, i in enumerate(insts):
            r = reqs[i]
            need[i] = len(r["hashes"]) - int(ml[j])
            st = self.stats[i]
            st[0] += 1
            st[1] += r["n_prompt"]
            st[2] += int(ml[j])
        # 4. eviction cascade
        decisions = {i: [] for i in insts}
        active = [i for i in insts if need[i] > len(self.free[i])]
        while active:
            k = np.zeros(self.n_inst, np.int32)
            for i in active:
                k[i] = min(max(need[i] - len(self.free[i]), self.k_min), self.max_k)
            dec = self.be.evict(now, k)
            nxt = []
            for i in active:
                d = dec[i]
                decisions[i].append(d)
                self.free[i].extend(d.tolist())
                self.stats[i][4] += len(d)
                self.stats[i][5] += 1
                if len(d) > 0 and need[i] > len(self.free[i]):
                    nxt.append(i)
            active = nxt
        # 5. insert the blocks after the match
        cols = {n: [] for n in ("inst", "ids", "hash", "parent", "types", "hints", "ob", "omax")}
        for j, i in enumerate(insts):
            r = reqs[i]
            m = int(ml[j])
            n = min(need[i], len(self.free[i]))
            self.stats[i][6] += need[i] - n
            self.stats[i][3] += n
            fr = self.free[i]
            ids = np.array([fr.pop() for _ in range(n)], np.int32)
            par = np.empty(n, np.int32)
            if n:
                par[0] = mids[j][m - 1] if m > 0 else -1
                par[1:] = ids[:-1]
            pos = np.arange(m, m + n, dtype=np.int32)
            cols["inst"].append(np.full(n, i, np.int32))
            cols["ids"].append(ids)
            cols["hash"].append(r["hashes"][m:m + n])
            cols["parent"].append(par)
            cols["types"].append(r["types"][m:m + n])
            cols["hints"].append(r["hints"][m:m + n])
            cols["ob"].append(pos)
            cols["omax"].append(np.full(n, len(r["hashes"]) - 1, np.int32))
            self.inflight[i].append(np.concatenate([np.asarray(mids[j], np.int32), ids]))
        flat = {n: np.concatenate(v) for n, v in cols.items()}
        if len(flat["ids"]):
            self.be.insert(now, flat)
            # 6. the running request holds its new blocks
            self.be.ref(flat["inst"], flat["ids"], +1)
        self.be.feedback()
        return {i: (int(ml[j]), decisions[i]) for j, i in enumerate(insts)}

    def summary(self, insts=None):
        insts = self.insts if insts is None else insts
        s = np.sum([self.stats[i] for i in insts], axis=0)
        return dict(requests=int(s[0]), prompt_blocks=int(s[1]), hit_blocks=int(s[2]), inserted=int(s[3]),
                    evicted=int(s[4]), decisions=int(s[5]), not_cached=int(s[6]),
                    block_hit_ratio=float(s[2]) / max(1, int(s[1])),
                    prefill_tokens=16 * (int(s[1]) - int(s[2])))
