"""TEST INFRASTRUCTURE — CPU oracle of SAECache's eviction hot path.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import
this module.  It shares no code with the HIP path and is deliberately plain:
full sorts, Python dicts and literal loops over the paper's rules.

One `OracleCache` object is one cache instance.  Its state follows the paper:

* a pool of KV blocks, each routed to a queue (Sec. 3.1, queue routing) with a
  token type tau(b) (Sec. 3.1: the type of the block's median token);
* the block index of the prefix cache: content hash -> block (strict prefix
  matching, Sec. 2.1);
* ``recently_evicted``: content hash -> (tau, queue) of recent victims
  (Algorithm 1, Add);
* ``token_stats[tau].{evicted, miss_after_evict}`` (Algorithm 3) and
  ``queue_hits[q]`` / ``queue_evictions[q]`` (Algorithm 2);
* the learned parameters w_tau, alpha_q, mu_q, sigma_q, gamma.

Readings of points where the paper is silent:

* A block is evictable iff it is valid, a leaf (no cached child) and
  unreferenced: tail-first eviction (Sec. 2.1 figure b) of free blocks.
* One eviction *decision* takes k victims from a snapshot: parameters and
  ``now`` are fixed, and a parent that becomes a leaf is eligible only at the
  next decision.  On a snapshot, k successive Evict() calls of Algorithm 1
  equal "stage 1 from the evict-first queue by (num_tokens, id), then stage 2
  by (P, id) over the other queues" (checked by `evict_sequential_literal`).
  Ties are broken by block id.
* ``recently_evicted`` keeps the victims of decision d while fewer than W
  evictions happened after d (W = ghost window).  An entry is consumed by
  the first Add() of its hash (counted once) and then forgotten.
* The learners run once per decision in which floor(evictions / K) grew
  (Algorithm 1's "every K evictions").  lambda = 0.99 decays a counter x to
  floor(99 x / 100) exactly.
* Algorithm 4 (online log-normal MLE) keeps one interval buffer per
  log-normal queue.  A prefix match that records intervals adds, for every
  request and every log-normal queue among its matched blocks, the elapsed
  time now - last_access of its deepest matched block of that queue, as it was
  before the call, when 1 <= dt < 2^31 ticks; a call's intervals join the buffer
  in request order.  The buffer keeps at most IVL_CAP intervals (the oldest
  leave first).  An update needs more than 20 intervals and then keeps the
  last 200 (Algorithm 4); mean and std are the population moments of the fp32
  ln of the intervals, summed exactly and rounded once (`sample_moments`).
* The decay-power learner (App. B) bins structural blocks by o_b / o_max into
  8 positional bins.  A bin's hit rate is hits / (hits + misses after
  eviction): prefix-match hits of blocks in the bin, and Add() calls that find
  a recently evicted block of the bin.  front = mean rate of bins 0-3, back =
  of bins 4-7 (bins without events left out); gamma moves by the EMA factor
  beta toward 1 / (back / front + 0.1) and is clipped to [0.3, 3.0].  It needs
  more than 20 events, events in both halves and front > 0; its counters
  restart after an update.  They are gathered only while the learner is on
  (the bin of an evicted block is always kept with its entry).
* The appendix text also states a token-weight rule (an EMA toward
  1 + 5 r_miss + 2 r_reuse) and a queue-weight rule (relative efficiency
  hits / capacity share, raised to 1/T); each is a learner of its own that
  replaces Algorithm 3, respectively 2, when chosen (`token_weights_ema`,
  `queue_weights_rel`, with their readings in their docstrings).
"""
import math

import numpy as np

from . import _native

EVICT_FIRST, STRUCTURAL, LOGNORMAL, RECENCY = 0, 1, 2, 3
N_TYPES = 5  # system, user, tool, response, cot — the order of Algorithm 3
N_BINS = 8   # positional bins of the decay-power learner
IVL_CAP = 4096  # intervals an Algorithm 4 buffer holds at most
F32 = np.float32
# Content hashes 0 and 2^64-1 are reserved by the boundary (they mark empty
# and deleted index slots there): Add() refuses a block that carries one, the
# index never holds one, so a request hash with one never matches.
RESERVED_HASHES = (0, 2 ** 64 - 1)


def block_type(counts):
    """tau(b) from per-block token-type counts [n, 5] (Sec. 3.1: the type of the
    median token).  Tokens are ranked by type in the order of Algorithm 3; the
    median is the lower median, rank floor((n-1)/2); tau is the type holding it."""
    counts = np.asarray(counts, np.int64)
    n = counts.sum(axis=1)
    m = (n - 1) // 2
    cum = np.cumsum(counts, axis=1)
    # first type whose cumulative count passes the median rank
    return np.argmax(cum > m[:, None], axis=1).astype(np.int32)


# Cache hint bits of a block (Algorithm 1's Classify reads them).
HINT_DECODE = 1         # decode-phase (generated) tokens
HINT_UNTEMPLATED = 2    # prefill content outside any shared template
HINT_MULTI_TURN = 4     # request is (or is predicted to be) multi-turn
HINT_AGENTIC = 8        # agentic / tool-use request
HINT_CONVERSATION = 16  # request carries a conversation id
HINT_SHARED_PREFIX = 32  # inside a prompt template shared across requests
# Queues Classify can return
ROLE_EVICT, ROLE_STRUCT, ROLE_CHAT, ROLE_AGENT = 0, 1, 2, 3
SYSTEM, COT = 0, 4


def classify_one(tau, hint):
    """Algorithm 1 Classify for one block: the first rule that holds, in the
    paper's order."""
    if tau == COT or hint & HINT_DECODE or hint & HINT_UNTEMPLATED:
        return ROLE_EVICT
    if hint & HINT_MULTI_TURN and hint & HINT_AGENTIC:
        return ROLE_AGENT
    if hint & HINT_MULTI_TURN or hint & HINT_CONVERSATION:
        return ROLE_CHAT
    if hint & HINT_SHARED_PREFIX or tau == SYSTEM:
        return ROLE_STRUCT
    return ROLE_EVICT


def classify(tau, hint, roles):
    """Queue index of every block: roles[Classify(tau, hint)]."""
    return np.array([roles[classify_one(int(t), int(h))] for t, h in zip(tau, hint)], np.int32)


def clamp(x, lo, hi):
    return min(max(x, F32(lo)), F32(hi))


class Params:
    """Learned parameters and learner settings (Sec. 3.1, App. B)."""

    def __init__(self, n_queues, w=1.0, alpha=1.0, mu=0.0, sigma=1.0, gamma=1.0,
                 eta=0.01, T=1.0, beta=0.1, K=32, learn_w=True, learn_alpha=True,
                 beta_ln=0.1, learn_ln=False, learn_gamma=False, learn_w_ema=False, learn_alpha_rel=False):
        def vec(v, n):
            a = np.zeros(n, F32)
            a[:] = np.resize(np.asarray(v, F32), n)
            return a
        self.w = vec(w, N_TYPES)
        self.alpha = vec(alpha, n_queues)
        self.mu = vec(mu, n_queues)
        self.sigma = vec(sigma, n_queues)
        self.gamma = F32(gamma)
        self.eta = F32(eta)
        self.T = F32(T)
        self.beta = F32(beta)
        self.K = int(K)
        self.learn_w = bool(learn_w)
        self.learn_alpha = bool(learn_alpha)
        self.beta_ln = F32(beta_ln)
        self.learn_ln = bool(learn_ln)
        self.learn_gamma = bool(learn_gamma)
        self.learn_w_ema = bool(learn_w_ema)
        self.learn_alpha_rel = bool(learn_alpha_rel)
        assert not (self.learn_w and self.learn_w_ema), "one token-weight rule at a time"
        assert not (self.learn_alpha and self.learn_alpha_rel), "one queue-weight rule at a time"


class OracleCache:
    def __init__(self, n_blocks, kinds, params, ghost_window=None):
        N = int(n_blocks)
        self.N = N
        self.kind = [int(k) for k in kinds]
        self.Q = len(self.kind)
        assert sum(k == EVICT_FIRST for k in self.kind) <= 1
        self.prm = params
        self.W = N if ghost_window is None else int(ghost_window)
        self.la = np.zeros(N, np.int32)
        self.queue = np.zeros(N, np.int32)
        self.tau = np.zeros(N, np.int32)
        self.ntok = np.full(N, 16, np.int32)
        self.ob = np.zeros(N, np.int32)
        self.omax = np.zeros(N, np.int32)
        self.valid = np.zeros(N, bool)
        self.ref_count = np.zeros(N, np.int32)
        self.child_count = np.zeros(N, np.int32)
        self.parent = np.full(N, -1, np.int32)
        self.hash = np.zeros(N, np.uint64)
        self.access_count = np.zeros(N, np.int32)
        self.index = {}
        self.ghost = {}
        self.evicted = [0] * N_TYPES
        self.missed = [0] * N_TYPES
        self.hits = [0] * self.Q
        self.evictions = [0] * self.Q
        self.ev_count = 0
        self.pending = False
        self.n_updates = 0
        self.ivl = [[] for _ in range(self.Q)]   # Algorithm 4 buffers (log-normal queues)
        self.bin_hits = [0] * N_BINS
        self.bin_missed = [0] * N_BINS
        self.type_hits = [0] * N_TYPES    # text-form token weights: hit blocks per type
        self.type_added = [0] * N_TYPES   # ... and blocks added per type

    # ------------------------------------------------------------------ state
    def bind(self, last_access, queue, tau, ntok, ob, omax, valid, ref_count,
             parent, hashes, access_count=None):
        """Set the whole pool; child counts follow from the parent links and the
        index holds every valid block (vLLM's prefix cache)."""
        self.la[:] = last_access
        self.queue[:] = queue
        self.tau[:] = tau
        self.ntok[:] = ntok
        self.ob[:] = ob
        self.omax[:] = omax
        self.valid[:] = np.asarray(valid, bool)
        self.ref_count[:] = ref_count
        self.parent[:] = parent
        self.hash[:] = hashes
        self.access_count[:] = 0 if access_count is None else access_count
        self.child_count[:] = 0
        has = self.valid & (self.parent >= 0)
        np.add.at(self.child_count, self.parent[has].astype(np.int64), 1)
        self.index = {int(self.hash[b]): b for b in np.nonzero(self.valid)[0].tolist()
                      if int(self.hash[b]) not in RESERVED_HASHES}

    def evictable(self):
        return self.valid & (self.child_count == 0) & (self.ref_count == 0)

    def ghost_live(self, entry):
        return self.ev_count - entry[2] < self.W

    def pos_bin(self, b):
        """Positional bin of block b: floor(8 o_b / o_max), o_b taken as at most
        o_max, bin 7 at the end and bin 0 for a one-block template (o_max = 0)."""
        omax = int(self.omax[b])
        if omax == 0:
            return 0
        o = min(int(self.ob[b]), omax)
        return min(N_BINS - 1, (N_BINS * o) // omax)

    # ---------------------------------------------------------- Eq. 1-3 keys
    def keys(self, now):
        p = self.prm
        return _native.score_blocks(now, self.la, self.queue, self.tau, self.ntok, self.ob,
                                    self.omax, self.kind, p.alpha, p.mu, p.sigma, p.w, p.gamma)

    # ------------------------------------------------- selection and decision
    def select_per_queue(self, now, k):
        """For every queue, the min(k, |evictable in q|) evictable blocks with the
        smallest (key, id), in that order."""
        key, p = self.keys(now)
        ev = self.evictable()
        lists = []
        for q in range(self.Q):
            ids = np.nonzero(ev & (self.queue == q))[0]
            order = np.lexsort((ids, key[ids]))
            lists.append(ids[order[:k]].astype(np.int32))
        return lists, key, p

    def decide(self, lists, key, k):
        """Algorithm 1 applied k times to one snapshot: stage 1 drains the
        evict-first queue by (num_tokens, id); stage 2 takes the rest by
        (P, id) over all other queues."""
        stage1 = np.zeros(0, np.int32)
        others = []
        for q in range(self.Q):
            if self.kind[q] == EVICT_FIRST:
                stage1 = lists[q][:k]
            else:
                others.append(lists[q])
        rest = k - len(stage1)
        cand = np.concatenate(others) if others else np.zeros(0, np.int32)
        order = np.lexsort((cand, key[cand]))
        stage2 = cand[order[:rest]]
        return np.concatenate([stage1, stage2]).astype(np.int32)

    def evict_sequential_literal(self, now, k):
        """Algorithm 1's Evict() called k times on one snapshot, written as the
        paper states it (strict '<' scan), blocks visited in id order."""
        key, _ = self.keys(now)
        P = key.view(np.float32)
        ev = self.evictable().copy()
        out = []
        for _ in range(k):
            ef = [q for q in range(self.Q) if self.kind[q] == EVICT_FIRST]
            victim = None
            if ef:
                best = None
                for b in range(self.N):
                    if ev[b] and self.queue[b] == ef[0]:
                        if best is None or self.ntok[b] < best:
                            best, victim = self.ntok[b], b
            if victim is None:
                best = math.inf
                for b in range(self.N):
                    if ev[b] and self.kind[self.queue[b]] != EVICT_FIRST:
                        if victim is None or P[b] < best:
                            best, victim = P[b], b
            if victim is None:
                break
            out.append(victim)
            ev[victim] = False
        return np.array(out, np.int32)

    def cascade_literal(self, now, k):
        """Algorithm 1's Evict() called k times on the live state (no
        snapshot): after each removal the victim's parent loses a child, and a
        parent left with none is evictable (valid, unreferenced, now a leaf)
        for the next call.  Written as the algorithm states it: every call
        rebuilds the evictable set and scans it (strict '<', blocks in id
        order).  Slow; for tiny pools."""
        key, _ = self.keys(now)
        P = key.view(np.float32)
        child = self.child_count.copy()
        gone = np.zeros(self.N, bool)
        ef = [q for q in range(self.Q) if self.kind[q] == EVICT_FIRST]
        out = []
        for _ in range(k):
            ev = self.valid & ~gone & (child == 0) & (self.ref_count == 0)
            victim = None
            if ef:
                best = None
                for b in range(self.N):
                    if ev[b] and self.queue[b] == ef[0] and (best is None or self.ntok[b] < best):
                        best, victim = self.ntok[b], b
            if victim is None:
                best = math.inf
                for b in range(self.N):
                    if ev[b] and self.kind[self.queue[b]] != EVICT_FIRST and (victim is None or P[b] < best):
                        best, victim = P[b], b
            if victim is None:
                break
            out.append(victim)
            gone[victim] = True
            if self.parent[victim] >= 0:
                child[self.parent[victim]] -= 1
        return np.array(out, np.int32)

    def decide_cascade(self, now, k):
        """The same sequence as `cascade_literal`, with two heaps: the
        evict-first queue by (num_tokens, id) and the other queues by
        (P, id); a parent whose last child leaves is pushed with its own key."""
        import heapq
        key, _ = self.keys(now)
        child = self.child_count.copy()
        ev = self.evictable()
        h1, h2 = [], []
        for b in np.nonzero(ev)[0].tolist():
            if self.kind[self.queue[b]] == EVICT_FIRST:
                h1.append((int(self.ntok[b]), b))
            else:
                h2.append((int(key[b]), b))
        heapq.heapify(h1)
        heapq.heapify(h2)
        out = []
        while len(out) < k and (h1 or h2):
            _, v = heapq.heappop(h1 if h1 else h2)
            out.append(v)
            par = int(self.parent[v])
            if par >= 0:
                child[par] -= 1
                if child[par] == 0 and self.valid[par] and self.ref_count[par] == 0:
                    if self.kind[self.queue[par]] == EVICT_FIRST:
                        heapq.heappush(h1, (int(self.ntok[par]), par))
                    else:
                        heapq.heappush(h2, (int(key[par]), par))
        return np.array(out, np.int32)

    def score_select(self, now, k, commit=False):
        lists, key, p = self.select_per_queue(now, k)
        decision = self.decide(lists, key, k)
        if commit:
            self.commit(decision)
        return lists, key, decision

    def commit(self, decision):
        """Remove the victims: index erase, recently_evicted insert (Algorithm 1),
        token_stats[tau].evicted++ (Algorithm 3), queue_evictions[q]++
        (Algorithm 2), and the parent becomes a leaf when its last child goes."""
        n = len(decision)
        before = self.ev_count
        stamp = before + n
        for b in decision.tolist():
            assert self.valid[b] and self.child_count[b] == 0 and self.ref_count[b] == 0
            self.valid[b] = False
            h = int(self.hash[b])
            if h not in RESERVED_HASHES:  # such a block was never indexed
                del self.index[h]
                self.ghost[h] = (int(self.tau[b]), int(self.queue[b]), stamp, self.pos_bin(b))
            self.evicted[self.tau[b]] += 1
            self.evictions[self.queue[b]] += 1
            par = int(self.parent[b])
            if par >= 0:
                self.child_count[par] -= 1
        self.ev_count = stamp
        K = self.prm.K
        if K > 0 and stamp // K > before // K:
            self.pending = True

    # ------------------------------------------------------------ prefix match
    def prefix_match(self, hashes, lens, now, touch=True, stats=True, intervals=False):
        """Strict prefix matching (Sec. 2.1): match_len = number of leading
        hashes found in the index.  All requests see the same snapshot; touches
        (last_access = now, access_count += 1 per request hit) apply afterwards.
        With stats, every hit block counts for queue_hits[queue(b)] and, in a
        structural queue with the decay-power learner on, for the hits of its
        positional bin.  With intervals,
        each request records Algorithm 4's reuse interval of each log-normal
        queue it hit: now - last_access of its deepest matched block there."""
        hashes = np.asarray(hashes, np.uint64)
        n = len(lens)
        mlen = np.zeros(n, np.int32)
        matched = np.full(hashes.shape, -1, np.int32)
        touched = []
        for r in range(n):
            m = 0
            while m < lens[r]:
                b = self.index.get(int(hashes[r, m]))
                if b is None:
                    break
                matched[r, m] = b
                m += 1
            mlen[r] = m
            deepest = {}
            for j in range(m):
                b = matched[r, j]
                q = int(self.queue[b])
                if stats:
                    self.hits[q] += 1
                    if self.kind[q] == STRUCTURAL and self.prm.learn_gamma:
                        self.bin_hits[self.pos_bin(b)] += 1
                    if self.prm.learn_w_ema:
                        self.type_hits[self.tau[b]] += 1
                if touch:
                    touched.append(b)
                if self.kind[q] == LOGNORMAL:
                    deepest[q] = b
            if intervals:
                for q in sorted(deepest):
                    dt = int(now) - int(self.la[deepest[q]])
                    if 1 <= dt < 2 ** 31:
                        buf = self.ivl[q]
                        buf.append(dt)
                        if len(buf) > IVL_CAP:
                            del buf[0]
        for b in touched:
            self.la[b] = now
            self.access_count[b] += 1
        return mlen, matched

    # ---------------------------------------------------------------- Add()
    def insert(self, ids, hashes, parent, last_access, queue, tau, ntok, ob, omax):
        """Algorithm 1 Add() for a batch of new blocks placed in free slots.
        A hash still in recently_evicted counts one miss after eviction for the
        type recorded at eviction, and leaves recently_evicted.  A block with a
        reserved hash is refused (not added, and its parent gains no child)."""
        refused = [int(h) in RESERVED_HASHES for h in np.asarray(hashes, np.uint64).tolist()]
        for i, b in enumerate(np.asarray(ids).tolist()):
            if refused[i]:
                continue
            assert not self.valid[b]
            h = int(hashes[i])
            assert h not in self.index
            self.valid[b] = True
            self.hash[b] = h
            self.parent[b] = parent[i]
            self.la[b] = last_access[i]
            self.queue[b] = queue[i]
            self.tau[b] = tau[i]
            self.ntok[b] = ntok[i]
            self.ob[b] = ob[i]
            self.omax[b] = omax[i]
            self.child_count[b] = 0
            self.ref_count[b] = 0
            self.access_count[b] = 0
            self.index[h] = b
            if self.prm.learn_w_ema:
                self.type_added[self.tau[b]] += 1
            g = self.ghost.pop(h, None)
            if g is not None and self.ghost_live(g):
                self.missed[g[0]] += 1
                if self.kind[g[1]] == STRUCTURAL and self.prm.learn_gamma:
                    self.bin_missed[g[3]] += 1
        for i in range(len(ids)):
            if parent[i] >= 0 and not refused[i]:
                self.child_count[parent[i]] += 1

    def ref(self, ids, delta):
        np.add.at(self.ref_count, np.asarray(ids, np.int64), int(delta))

    # ------------------------------------------------------------- learners
    def token_weights(self):
        """Algorithm 3, in fp32.  Per type: when more than ten of its blocks
        have been evicted, the weight is multiplied by 1 + eta * r, r the
        share of those evictions that were asked for again, and clamped to
        [0.1, 5]; both counts then lose 1 % (lambda = 0.99 as floor(99 x / 100))
        whether or not the weight moved."""
        p = self.prm
        for t in range(N_TYPES):
            ev, mi = self.evicted[t], self.missed[t]
            if ev > 10:
                returns_per_eviction = F32(mi) / F32(ev)
                p.w[t] = clamp(p.w[t] * (F32(1.0) + p.eta * returns_per_eviction), 0.1, 5.0)
            self.evicted[t], self.missed[t] = (99 * ev) // 100, (99 * mi) // 100

    def queue_weights(self):
        """Algorithm 2, in fp32, for every queue but the evict-first one: with
        more than five evictions since the last run, alpha moves the fraction
        beta of the way to 1 + (hits per eviction) / T and is clamped to
        [0.1, 3]; the queue's hit and eviction counts restart in any case."""
        p = self.prm
        for q in range(self.Q):
            if self.kind[q] == EVICT_FIRST:
                continue
            h, e = self.hits[q], self.evictions[q]
            if e > 5:
                goal = F32(1.0) + (F32(h) / F32(e)) / p.T
                p.alpha[q] = clamp(p.alpha[q] + p.beta * (goal - p.alpha[q]), 0.1, 3.0)
            self.hits[q], self.evictions[q] = 0, 0

    def token_weights_ema(self):
        """The appendix text's token-weight rule (App. B): per type,
        w_target = 1 + 5 r_miss + 2 r_reuse and w <- (1 - eta) w + eta w_target,
        in fp32.  r_miss = missed / evicted (0 without evictions); r_reuse = hit
        blocks / (hit blocks + blocks added), the type's cache hit rate (0
        without either).  All four counters decay by 0.99 (floored) per run;
        w stays in Algorithm 3's [0.1, 5.0]."""
        p = self.prm
        one = F32(1.0)
        for t in range(N_TYPES):
            ev, mi = self.evicted[t], self.missed[t]
            h, a = self.type_hits[t], self.type_added[t]
            r_miss = F32(mi) / F32(ev) if ev > 0 else F32(0.0)
            r_reuse = F32(h) / F32(h + a) if h + a > 0 else F32(0.0)
            target = one + r_miss * F32(5.0) + r_reuse * F32(2.0)
            p.w[t] = clamp((one - p.eta) * p.w[t] + p.eta * target, 0.1, 5.0)
            self.evicted[t] = (99 * ev) // 100
            self.missed[t] = (99 * mi) // 100
            self.type_hits[t] = (99 * h) // 100
            self.type_added[t] = (99 * a) // 100

    def resident(self):
        """Cached (valid) blocks per queue."""
        return [int(np.count_nonzero(self.valid & (self.queue == q))) for q in range(self.Q)]

    def queue_weights_rel(self):
        """The appendix text's queue-weight rule (App. B): E_q = H_q / C_q
        with H_q the queue's hit blocks since the last run and C_q its share of
        the cached blocks; alpha_q <- beta alpha_q + (1 - beta) (E_q / E_mean)^(1/T)
        over the queues but the evict-first one that hold blocks, E_mean their
        mean, in fp32 (x^(1/T) = exp(ln x / T) in the fp32 recipe, x itself for
        T = 1); clamped to Algorithm 2's [0.1, 3.0].  Runs only when E_mean > 0;
        hits and evictions restart after every run."""
        p = self.prm
        res = self.resident()
        total = sum(res)
        qs = [q for q in range(self.Q) if self.kind[q] != EVICT_FIRST and res[q] > 0]
        if total > 0 and qs:
            E = {}
            for q in qs:
                share = F32(res[q]) / F32(total)
                E[q] = F32(self.hits[q]) / share
            e_sum = F32(0.0)
            for q in qs:
                e_sum = e_sum + E[q]
            e_mean = e_sum / F32(len(qs))
            if e_mean > 0:
                for q in qs:
                    x = E[q] / e_mean
                    if p.T == F32(1.0) or x == 0:
                        tgt = x
                    else:
                        lx = _native.ln(np.array([x], F32))[0]
                        tgt = _native.exp(np.array([lx / p.T], F32))[0]
                    p.alpha[q] = clamp(p.beta * p.alpha[q] + (F32(1.0) - p.beta) * tgt, 0.1, 3.0)
        for q in range(self.Q):
            if self.kind[q] != EVICT_FIRST:
                self.hits[q] = 0
                self.evictions[q] = 0

    def lognormal_params(self):
        """Algorithm 4 for every log-normal queue (one estimator per queue)."""
        p = self.prm
        for q in range(self.Q):
            if self.kind[q] != LOGNORMAL:
                continue
            buf = self.ivl[q]
            if len(buf) > 20:
                mu_s, sigma_s = sample_moments(buf)
                p.mu[q] = p.mu[q] + p.beta_ln * (mu_s - p.mu[q])
                s = p.sigma[q] + p.beta_ln * (sigma_s - p.sigma[q])
                p.sigma[q] = max(s, F32(0.1))
                self.ivl[q] = buf[-200:]

    def decay_power(self):
        """Decay-power learner (App. B) over the 8 positional bins."""
        p = self.prm
        events = [self.bin_hits[i] + self.bin_missed[i] for i in range(N_BINS)]
        if sum(events) <= 20:
            return
        rates = [F32(self.bin_hits[i]) / F32(events[i]) if events[i] else None for i in range(N_BINS)]
        half = N_BINS // 2
        front = [r for r in rates[:half] if r is not None]
        back = [r for r in rates[half:] if r is not None]
        if not front or not back:
            return
        f_avg = F32(0.0)
        for r in front:
            f_avg = f_avg + r
        f_avg = f_avg / F32(len(front))
        b_avg = F32(0.0)
        for r in back:
            b_avg = b_avg + r
        b_avg = b_avg / F32(len(back))
        if not f_avg > 0:
            return
        ratio = b_avg / f_avg
        est = F32(1.0) / (ratio + F32(0.1))
        p.gamma = clamp(p.gamma + p.beta * (est - p.gamma), 0.3, 3.0)
        self.bin_hits = [0] * N_BINS
        self.bin_missed = [0] * N_BINS

    def feedback(self, force=False):
        if not (self.pending or force):
            return False
        if self.prm.learn_w:
            self.token_weights()
        if self.prm.learn_w_ema:
            self.token_weights_ema()
        if self.prm.learn_alpha:
            self.queue_weights()
        if self.prm.learn_alpha_rel:
            self.queue_weights_rel()
        if self.prm.learn_ln:
            self.lognormal_params()
        if self.prm.learn_gamma:
            self.decay_power()
        self.pending = False
        self.n_updates += 1
        return True

    def counters(self):
        return dict(evicted=list(self.evicted), missed=list(self.missed),
                    hits=list(self.hits), evictions=list(self.evictions),
                    ev_count=self.ev_count, pending=self.pending,
                    bin_hits=list(self.bin_hits), bin_missed=list(self.bin_missed),
                    type_hits=list(self.type_hits), type_added=list(self.type_added),
                    resident=self.resident())


def sample_moments(intervals):
    """Algorithm 4's mu_sample, sigma_sample: mean and population std of
    ln(dt) over the buffer.  ln is the fp32 recipe's ln of fl32(dt).  Every
    x = ln(dt) is 0 or at least ln 2, so X = x * 2^24 is an integer and the
    sums S1 = sum X, S2 = sum X^2 are exact; then, in IEEE double,
    m = S1 / n * 2^-24, v = max(S2 / n * 2^-48 - m * m, 0), with S2 converted
    as hi * 2^64 + lo (hi, lo its 64-bit halves), and the results rounded to
    fp32: mu = fl32(m), sigma = fl32(sqrt(v))."""
    x = _native.ln(np.asarray(intervals, np.float64).astype(F32))
    n = len(x)
    X = [int(F32(v).astype(np.float64) * 2.0 ** 24) for v in x]
    assert all(float(Xi) == float(v) * 2.0 ** 24 for Xi, v in zip(X, x))
    S1 = sum(X)
    S2 = sum(Xi * Xi for Xi in X)
    m = (float(S1) / float(n)) * 2.0 ** -24
    s2 = float(S2 >> 64) * 2.0 ** 64 + float(S2 & (2 ** 64 - 1))
    v = (s2 / float(n)) * 2.0 ** -48 - m * m
    if v < 0.0:
        v = 0.0
    return F32(m), F32(math.sqrt(v))
