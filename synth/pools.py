"""Seeded block pools, hash chains and prefix-match request batches.

Workload recipe (the paper's own workloads are real traces that are not
available; these draws stand in for them with the shapes the configurations
state):

* token-type counts per 16-token block: Dirichlet(0.5) over the 5 types
  scaled to 16, rounded by largest remainder (ties to the lower type index);
* last_access ~ U{0 .. 999,999} ms ticks, evaluated at now = 1,000,000;
* access_count ~ Geometric(0.3); 30 % of blocks non-leaf, 10 % referenced;
* queue mix per configuration; o_max ~ U{31 .. 250} blocks (500 - 4,000
  token templates in 16-token blocks), o_b ~ U{0 .. o_max};
* log-normal parameters from Table 3 (chat mu 4.82 s / sigma 1.25, agent
  mu 2.28 s / sigma 1.34), moved to ms ticks by + ln 1000;
* leafness is drawn per block as stated; parent links are made consistent
  with it: each non-leaf block parents exactly one distinct leaf block, so an
  eviction can turn its parent into a leaf;
* block hashes form chains h_i = mix64(h_{i-1} xor c_i) with random 64-bit
  content ids c_i (mix64 = the SplitMix64 finalizer of Steele, Lea & Flood,
  2014); block b holds position b mod L of chain b div L;
* requests: length U{1 .. max_len}; 60 % start with a prefix (length
  U{1 .. len}) of a random chain and continue with fresh content, the rest are
  fresh from the first block.
"""
import math

import numpy as np

LN_1000 = math.log(1000.0)
MU_CHAT_MS = 4.82 + LN_1000
SIGMA_CHAT = 1.25
MU_AGENT_MS = 2.28 + LN_1000
SIGMA_AGENT = 1.34

EF, STRUCT, LN, REC = 0, 1, 2, 3
NOW = 1_000_000
ROOT = np.uint64(0x243F6A8885A308D3)  # fixed chain root (hex digits of pi)
M64 = (1 << 64) - 1

CONFIGS = {
    # 3 queues: session (log-normal, chat timing), template (structural), default (recency)
    "tiny": dict(n_blocks=4096, kinds=[LN, STRUCT, REC], mix=[0.50, 0.35, 0.15],
                 mu=[MU_CHAT_MS, 0.0, 0.0], sigma=[SIGMA_CHAT, 1.0, 1.0],
                 k=64, chain_len=32, n_req=256, req_len=32, hit_frac=0.6, seed=1001),
    "mid": dict(n_blocks=262144, kinds=[LN, STRUCT, REC], mix=[0.50, 0.35, 0.15],
                mu=[MU_CHAT_MS, 0.0, 0.0], sigma=[SIGMA_CHAT, 1.0, 1.0],
                k=1024, chain_len=32, n_req=256, req_len=32, hit_frac=0.6, seed=1002,
                n_decisions=64, rerequest=0.05),
    # 5 queues: evict-first, structural, chat, agent, default
    "large": dict(n_blocks=4194304, kinds=[EF, STRUCT, LN, LN, REC],
                  mix=[0.10, 0.30, 0.30, 0.20, 0.10],
                  mu=[0.0, 0.0, MU_CHAT_MS, MU_AGENT_MS, 0.0],
                  sigma=[1.0, 1.0, SIGMA_CHAT, SIGMA_AGENT, 1.0],
                  k=4096, chain_len=128, n_req=4096, req_len=128, hit_frac=0.6, seed=1004),
}


def pool_config(name, **over):
    c = dict(CONFIGS[name])
    c.update(over)
    return c


def mix64(z):
    """SplitMix64 finalizer on uint64 arrays (wrapping arithmetic)."""
    z = np.asarray(z, np.uint64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        z = z ^ (z >> np.uint64(31))
    return z


def _fix_reserved(h):
    """0 marks an empty index slot and 2^64-1 a deleted one: remap both to 1."""
    h = h.copy()
    h[(h == np.uint64(0)) | (h == np.uint64(M64))] = np.uint64(1)
    return h


def _rand_u64(rng, shape):
    return rng.integers(0, M64, size=shape, dtype=np.uint64, endpoint=True)


def chain_hashes(n_chains, L, rng):
    """[n_chains, L] chained hashes from random content ids."""
    c = _rand_u64(rng, (n_chains, L))
    out = np.empty((n_chains, L), np.uint64)
    h = np.full(n_chains, ROOT, np.uint64)
    for i in range(L):
        h = _fix_reserved(mix64(h ^ c[:, i]))
        out[:, i] = h
    return out


def token_type_counts(rng, n, tokens=16, conc=0.5):
    """Dirichlet(conc) type shares scaled to `tokens`, largest-remainder rounding."""
    d = rng.dirichlet(np.full(5, conc), size=n)
    x = d * tokens
    fl = np.floor(x).astype(np.int64)
    rem = tokens - fl.sum(axis=1)
    frac = x - fl
    order = np.argsort(-frac, axis=1, kind="stable")
    rank = np.empty_like(order)
    np.put_along_axis(rank, order, np.arange(5)[None, :].repeat(n, 0), axis=1)
    fl += (rank < rem[:, None]).astype(np.int64)
    return fl.astype(np.uint8)


def make_pool(cfg, seed=None, n_blocks=None):
    """A full pool of one instance, as plain numpy arrays."""
    N = int(n_blocks or cfg["n_blocks"])
    seed = cfg["seed"] if seed is None else seed
    rs = [np.random.Generator(np.random.PCG64(s)) for s in np.random.SeedSequence(seed).spawn(10)]
    Q = len(cfg["kinds"])
    counts = token_type_counts(rs[0], N)
    last_access = rs[1].integers(0, NOW, size=N, dtype=np.int64).astype(np.int32)
    access_count = rs[2].geometric(0.3, size=N).astype(np.int32)
    queue = rs[3].choice(Q, size=N, p=np.asarray(cfg["mix"]) / np.sum(cfg["mix"])).astype(np.int32)
    omax = rs[4].integers(31, 251, size=N).astype(np.int32)
    ob = (rs[4].random(N) * (omax + 1)).astype(np.int32)
    ob = np.minimum(ob, omax)
    nonleaf = rs[5].random(N) < 0.3
    ref_count = (rs[6].random(N) < 0.1).astype(np.int32)
    parent = np.full(N, -1, np.int32)
    nl = np.nonzero(nonleaf)[0]
    leaves = np.nonzero(~nonleaf)[0]
    kids = rs[7].choice(leaves, size=min(len(nl), len(leaves)), replace=False)
    parent[kids] = nl[:len(kids)]
    L = int(cfg["chain_len"])
    n_chains = (N + L - 1) // L
    chains = chain_hashes(n_chains, L, rs[8])
    hashes = chains.reshape(-1)[:N].copy()
    return dict(
        n_blocks=N, now=NOW, counts=counts, last_access=last_access,
        access_count=access_count, queue=queue, ntok=np.full(N, 16, np.int32),
        ob=ob, omax=omax, valid=np.ones(N, bool), ref_count=ref_count,
        parent=parent, hash=hashes, chains=chains, seed=seed,
    )


def make_requests(chains, n_req, max_len, hit_frac, rng_or_seed):
    """[n_req, max_len] request hashes (0 past each length) and lengths."""
    rng = (rng_or_seed if isinstance(rng_or_seed, np.random.Generator)
           else np.random.Generator(np.random.PCG64(np.random.SeedSequence(rng_or_seed))))
    n_chains, L = chains.shape
    lens = rng.integers(1, max_len + 1, size=n_req).astype(np.int32)
    hit = rng.random(n_req) < hit_frac
    cidx = rng.integers(0, n_chains, size=n_req)
    m = np.minimum((rng.random(n_req) * lens).astype(np.int64) + 1, np.minimum(lens, L))
    fresh = _rand_u64(rng, (n_req, max_len))
    out = np.zeros((n_req, max_len), np.uint64)
    h = np.full(n_req, ROOT, np.uint64)
    for j in range(max_len):
        from_chain = hit & (j < m)
        ch = chains[cidx, min(j, L - 1)]
        hj = np.where(from_chain, ch, _fix_reserved(mix64(h ^ fresh[:, j])))
        hj = np.where(j < lens, hj, np.uint64(0))
        out[:, j] = hj
        h = hj
    return out, lens
