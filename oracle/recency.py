"""TEST INFRASTRUCTURE — per-(queue, type) recency lists: a faster exact CPU
selection (the per-queue heap idea of the paper's cost discussion, Sec. 3.2 and
Algorithm 1), used as a second CPU baseline beside the oracle.

Only tests/ and bench.py's cpu_baseline leg use it; it shares no code with
the HIP path.  It reads a bound OracleCache's snapshot and gives the same per-queue
lists and decision as OracleCache.select_per_queue / decide:

* log-normal and recency queues: one list per (queue, type) of evictable
  blocks in (last_access, id) order, walked from the oldest block with the
  stopping rule of recency.c (P along such a list never rises by more than a
  factor 1 + 2^-19 in the fp32 recipe);
* evict-first queue: one list in (num_tokens, id) order, whose first k blocks
  are the answer (the key is num_tokens);
* structural queue: P also depends on o_b / o_max, so every evictable block
  of the queue is scored into a bounded heap.

Building the lists stands for their upkeep in a live cache (a block moves to
the tail of its list when touched, joins at insert and leaves at eviction, all
O(1) while time only grows); `build` is timed apart from `select`.
"""
import numpy as np

from . import _native
from .policy import EVICT_FIRST, LOGNORMAL, N_TYPES, RECENCY, STRUCTURAL


class RecencyLists:
    def __init__(self, cache):
        self.c = cache
        self.build()

    def build(self):
        c = self.c
        ev = c.evictable()
        self.groups = {}
        for q in range(c.Q):
            ids = np.nonzero(ev & (c.queue == q))[0].astype(np.int32)
            kind = c.kind[q]
            if kind in (LOGNORMAL, RECENCY):
                tau = c.tau[ids]
                order = np.lexsort((ids, c.la[ids], tau))  # by type, then (last_access, id)
                gids = np.ascontiguousarray(ids[order])
                start = np.searchsorted(tau[order], np.arange(N_TYPES + 1)).astype(np.int64)
                self.groups[q] = (gids, start)
            elif kind == EVICT_FIRST:
                self.groups[q] = np.ascontiguousarray(ids[np.lexsort((ids, c.ntok[ids]))])
            else:
                self.groups[q] = np.ascontiguousarray(ids)
        self.visited = 0

    def select_per_queue(self, now, k, prefill=None):
        """Per queue, the min(k, evictable) smallest (key, id); also the keys of
        the listed blocks (bits of P, or of (float) num_tokens).  prefill: blocks
        per list scored before the walk (k by default; any value is exact)."""
        c, prm = self.c, self.c.prm
        L = _native.lib()
        p = _native._ptr
        lists, keys = [], []
        heap = np.empty(max(k, 1), np.uint64)
        self.visited = 0
        la = np.ascontiguousarray(c.la, np.int32)
        for q in range(c.Q):
            kind = c.kind[q]
            out_k = np.empty(max(k, 1), np.uint32)
            out_i = np.empty(max(k, 1), np.int32)
            aw = np.ascontiguousarray(np.float32(prm.alpha[q]) * prm.w.astype(np.float32), np.float32)
            if kind in (LOGNORMAL, RECENCY):
                gids, start = self.groups[q]
                vis = np.zeros(1, np.int64)
                pf = k if prefill is None else prefill
                n = L.oracle_rl_select(int(k), int(pf), int(now), int(kind), float(prm.mu[q]), float(prm.sigma[q]),
                                       p(aw), p(start), p(gids), p(la), p(heap), p(out_k), p(out_i), p(vis))
                self.visited += int(vis[0])
            elif kind == STRUCTURAL:
                ids = self.groups[q]
                n = L.oracle_struct_select(int(k), int(now), float(prm.gamma), p(aw), ids.size, p(ids), p(la),
                                           p(np.ascontiguousarray(c.tau, np.int32)),
                                           p(np.ascontiguousarray(c.ob, np.int32)),
                                           p(np.ascontiguousarray(c.omax, np.int32)), p(heap), p(out_k), p(out_i))
                self.visited += ids.size
            else:  # evict-first: (num_tokens, id) order is the key order
                ids = self.groups[q][:k]
                n = ids.size
                out_i[:n] = ids
                out_k[:n] = c.ntok[ids].astype(np.float32).view(np.uint32)
            lists.append(out_i[:n].copy())
            keys.append(out_k[:n].copy())
        return lists, keys

    def decide(self, lists, keys, k):
        """Algorithm 1 applied k times to the snapshot (as OracleCache.decide)."""
        stage1 = np.zeros(0, np.int32)
        cand, ckey = [], []
        for q in range(self.c.Q):
            if self.c.kind[q] == EVICT_FIRST:
                stage1 = lists[q][:k]
            else:
                cand.append(lists[q])
                ckey.append(keys[q])
        rest = k - len(stage1)
        cand = np.concatenate(cand) if cand else np.zeros(0, np.int32)
        ckey = np.concatenate(ckey) if ckey else np.zeros(0, np.uint32)
        order = np.lexsort((cand, ckey))
        return np.concatenate([stage1, cand[order[:rest]]]).astype(np.int32)

    def score_select(self, now, k, prefill=None):
        lists, keys = self.select_per_queue(now, k, prefill)
        return lists, keys, self.decide(lists, keys, k)
