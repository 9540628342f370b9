// Block index, recently_evicted, prefix matching, Add() and eviction commit.
//
// Block index: open addressing, linear probing, 16-byte slots {hash, id} in
// HBM; 0 marks an empty slot and 2^64-1 a deleted one.  Lookups run in
// kernels that never write the index, so every request of a prefix-match batch
// sees the same index.
//
// recently_evicted (Algorithm 1): victims are appended to a ring of
// W + max_k entries in eviction order, each stamped with the eviction count
// right after its decision; an entry is live while fewer than W evictions
// followed it.  A hash table maps a content hash to its ring position; a
// lookup follows a slot only if the ring entry there still holds that hash,
// is live and not consumed.  A reused ring slot's old table slot is therefore
// left in place (stale, like a deleted one) and the table is rebuilt from the
// ring once stale and deleted slots reach a quarter of it, so a commit only
// inserts.
#include "sae_internal.h"
#include "pm_match.h"

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ bool index_insert(IndexSlot *tab, uint32_t mask, unsigned long long h, int32_t id,
                                             uint32_t tq)
{
    uint32_t s = hash_home(h, mask);
    for (int p = 0; p <= (int)mask && p < SAE_MAX_PROBES; ++p) {
        unsigned long long v = tab[s].hash;
        if (v == SAE_EMPTY_HASH || v == SAE_TOMB_HASH) {
            unsigned long long old = atomicCAS(&tab[s].hash, v, h);
            if (old == v) {
                *reinterpret_cast<uint2 *>(&tab[s].id) = make_uint2((uint32_t)id, tq);
                return true;
            }
            continue;  // lost the slot: look at it again
        }
        s = (s + 1) & mask;
    }
    return false;
}

// index_insert with the home slot's hash already loaded, and the lookup of a
// live, unconsumed recently_evicted entry of hash h (its table slot index, or
// -1; *ring_pos its ring position) likewise.
__device__ __forceinline__ bool index_insert_from(IndexSlot *tab, uint32_t mask, unsigned long long h, int32_t id,
                                                  uint32_t tq, uint32_t s0, unsigned long long v0)
{
    uint32_t s = s0;
    unsigned long long v = v0;
    bool fresh = true;  // v holds slot s's hash as loaded
    for (int p = 0; p <= (int)mask && p < SAE_MAX_PROBES; ++p) {
        if (!fresh) v = tab[s].hash;
        fresh = false;
        if (v == SAE_EMPTY_HASH || v == SAE_TOMB_HASH) {
            const unsigned long long old = atomicCAS(&tab[s].hash, v, h);
            if (old == v) {
                *reinterpret_cast<uint2 *>(&tab[s].id) = make_uint2((uint32_t)id, tq);
                return true;
            }
            continue;  // lost the slot: look at it again
        }
        s = (s + 1) & mask;
    }
    return false;
}

__device__ __forceinline__ int ghost_find_from(const GhostSlot *tab, uint32_t mask, const GhostEntry *ring,
                                               unsigned long long h, long long ev_now, int W, uint32_t s0,
                                               unsigned long long v0, uint32_t *ring_pos)
{
    if (SAE_HASH_RESERVED(h)) return -1;
    uint32_t s = s0;
    for (int p = 0; p <= (int)mask && p < SAE_MAX_PROBES; ++p) {
        const unsigned long long v = p == 0 ? v0 : tab[s].hash;
        if (v == SAE_EMPTY_HASH) return -1;
        if (v == h) {
            const uint32_t r = tab[s].ring;
            const GhostEntry &g = ring[r];
            if (g.hash == h && !(g.tq & SAE_TQ_CONSUMED) && ev_now - g.stamp < (long long)W) {
                *ring_pos = r;
                return (int)s;
            }
        }
        s = (s + 1) & mask;
    }
    return -1;
}

__device__ __forceinline__ bool ghost_insert(GhostSlot *tab, uint32_t mask, unsigned long long h, uint32_t ring_pos)
{
    uint32_t s = hash_home(h, mask);
    for (int p = 0; p <= (int)mask && p < SAE_MAX_PROBES; ++p) {
        unsigned long long v = tab[s].hash;
        if (v == SAE_EMPTY_HASH || v == SAE_TOMB_HASH) {
            unsigned long long old = atomicCAS(&tab[s].hash, v, h);
            if (old == v) {
                tab[s].ring = ring_pos;
                return true;
            }
            continue;
        }
        s = (s + 1) & mask;
    }
    return false;
}

// ---------------------------------------------------------------------------
// tau(b): type holding the lower-median token when tokens are ranked by type.
__global__ void k_block_type(const uint8_t *counts, long long n, uint8_t *tau)
{
    long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const uint8_t *cb = counts + i * SAE_N_TYPES;
    int total = 0;
    for (int t = 0; t < SAE_N_TYPES; ++t) total += cb[t];
    int m = (total - 1) >> 1;  // total >= 1 expected; total 0 gives type 0
    int run = 0, ty = 0;
    for (int t = 0; t < SAE_N_TYPES; ++t) {
        run += cb[t];
        if (run > m) {
            ty = t;
            break;
        }
    }
    tau[i] = (uint8_t)ty;
}

// Algorithm 1 Classify: queue of a block from its hints and its type.
__global__ void k_classify(int n, const uint8_t *hint, uint16_t *meta, int r_evict, int r_struct, int r_chat,
                           int r_agent)
{
    int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    unsigned h = hint[i];
    unsigned m = meta[i];
    unsigned tau = (unsigned)meta_type(m);
    int q;
    if (tau == SAE_TYPE_COT || (h & (SAE_HINT_DECODE | SAE_HINT_UNTEMPLATED))) q = r_evict;
    else if ((h & SAE_HINT_MULTI_TURN) && (h & SAE_HINT_AGENTIC)) q = r_agent;
    else if (h & (SAE_HINT_MULTI_TURN | SAE_HINT_CONVERSATION)) q = r_chat;
    else if ((h & SAE_HINT_SHARED_PREFIX) || tau == SAE_TYPE_SYSTEM) q = r_struct;
    else q = r_evict;
    meta[i] = (uint16_t)((m & ~7u) | (unsigned)q);
}

// Clear index, recently_evicted and counters.
__global__ void k_clear_all(DevCtx c, int clear_ghost_and_counters)
{
    long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    long long nidx = (long long)c.n_inst * ((long long)c.index_mask + 1);
    if (i < nidx) {
        c.index[i].hash = SAE_EMPTY_HASH;
        c.index[i].id = -1;
        c.index[i].tq = 0;
    }
    if (!clear_ghost_and_counters) return;
    long long ngt = (long long)c.n_inst * ((long long)c.ghost_mask + 1);
    if (i < ngt) {
        c.gtab[i].hash = SAE_EMPTY_HASH;
        c.gtab[i].ring = 0;
    }
    long long nring = (long long)c.n_inst * c.ring_cap;
    if (i < nring) {
        c.ring[i].hash = 0;
        c.ring[i].stamp = 0;
        c.ring[i].tq = 0;
    }
    long long ncp = (long long)c.n_inst * SAE_CSLOTS * SAE_CF_STRIDE;
    if (i < ncp) c.cpart[i] = 0;
    if (i < c.n_inst) {
        InstState &s = c.state[i];
        for (int t = 0; t < SAE_N_TYPES; ++t) s.evicted[t] = s.missed[t] = 0;
        for (int q = 0; q < SAE_MAX_QUEUES; ++q) s.hits[q] = s.evictions[q] = 0;
        s.ev_count = 0;
        s.ev_before = 0;
        s.pending = 0;
        s.n_updates = 0;
        s.last_d = 0;
        for (int b = 0; b < SAE_N_BINS; ++b) s.bin_hits[b] = s.bin_missed[b] = 0;
        for (int t = 0; t < SAE_N_TYPES; ++t) s.type_hits[t] = s.type_added[t] = 0;
        for (int q = 0; q < SAE_MAX_QUEUES; ++q) s.ivl_n[q] = s.ivl_start[q] = s.resident[q] = 0;
    }
}

// Insert every valid block's hash into its instance's index and, on a full
// build (`census`), count the cached blocks per queue (summed per workgroup in
// LDS when the workgroup lies in one instance).  A rebuild of the index alone
// leaves the counts, which commits and Add() keep current.
__global__ void k_index_fill(DevCtx c, int census)
{
    __shared__ int32_t cnt[SAE_MAX_QUEUES];
    if (threadIdx.x < SAE_MAX_QUEUES) cnt[threadIdx.x] = 0;
    __syncthreads();
    const long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    const long long total = (long long)c.n_inst * c.N;
    const long long g0 = (long long)blockIdx.x * blockDim.x;
    const long long g1 = (g0 + blockDim.x < total ? g0 + blockDim.x : total) - 1;
    const int i0 = (int)(g0 / c.N);
    const bool one_inst = (int)(g1 / c.N) == i0;
    if (g < total) {
        const uint32_t m = c.meta[g];
        if (m & SAE_META_VALID) {
            const int inst = (int)(g / c.N);
            const int32_t b = (int32_t)(g - (long long)inst * c.N);
            IndexSlot *tab = c.index + (long long)inst * ((long long)c.index_mask + 1);
            const unsigned long long h = c.hash[g];
            if (SAE_HASH_RESERVED(h)) set_status(c.status, SAE_ST_BAD_HASH);
            else if (!index_insert(tab, c.index_mask, h, b, slot_tq(m, c.off[g])))
                set_status(c.status, SAE_ST_INDEX_FULL);
            if (census) {
                if (one_inst) atomicAdd(&cnt[meta_queue(m)], 1);
                else atomicAdd(counter_slot(c, inst, blockIdx.x) + SAE_CF_RES + meta_queue(m), 1);
            }
        }
    }
    __syncthreads();
    if (census && one_inst && threadIdx.x < SAE_MAX_QUEUES && cnt[threadIdx.x])
        atomicAdd(counter_slot(c, i0, blockIdx.x) + SAE_CF_RES + threadIdx.x, cnt[threadIdx.x]);
}

// Rebuild recently_evicted from the ring (drops tombstones).
__global__ void k_ghost_clear(DevCtx c)
{
    long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    long long ngt = (long long)c.n_inst * ((long long)c.ghost_mask + 1);
    if (i < ngt) c.gtab[i].hash = SAE_EMPTY_HASH;
}
__global__ void k_ghost_fill(DevCtx c)
{
    long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    long long nring = (long long)c.n_inst * c.ring_cap;
    if (i >= nring) return;
    int inst = (int)(i / c.ring_cap);
    uint32_t r = (uint32_t)(i - (long long)inst * c.ring_cap);
    GhostEntry g = c.ring[i];
    if (g.hash == 0 || (g.tq & SAE_TQ_CONSUMED)) return;
    if (c.state[inst].ev_count - g.stamp >= (long long)c.W) return;
    GhostSlot *tab = c.gtab + (long long)inst * ((long long)c.ghost_mask + 1);
    if (!ghost_insert(tab, c.ghost_mask, g.hash, r)) set_status(c.status, SAE_ST_GHOST_FULL);
}

// ---------------------------------------------------------------------------
// Add(), phase 1: write the block, index it, consume its recently_evicted entry.
__global__ void k_insert_a(DevCtx c, int n, const int32_t *inst_a, const int32_t *ids, const uint64_t *hash,
                           const int32_t *parent, const int32_t *la, const uint16_t *meta, const uint32_t *off,
                           uint8_t *skip)
{
    int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    int inst = inst_a ? inst_a[i] : 0;
    int32_t b = ids[i];
    const unsigned long long h = hash[i];
    const bool ok = inst >= 0 && inst < c.n_inst && b >= 0 && b < c.N;
    // the slot's meta and the first probes of the index and of recently_evicted
    // go out together (addresses clamped into the instance's tables)
    const int ic = ok ? inst : 0;
    const long long g = (long long)ic * c.N + (ok ? b : 0);
    IndexSlot *tab = c.index + (long long)ic * ((long long)c.index_mask + 1);
    GhostSlot *gt = c.gtab + (long long)ic * ((long long)c.ghost_mask + 1);
    GhostEntry *ring = c.ring + (long long)ic * c.ring_cap;
    const uint32_t si = hash_home(h, c.index_mask), sg = hash_home(h, c.ghost_mask);
    const uint32_t mg = c.meta[g];
    const unsigned long long vi = tab[si].hash, vg = gt[sg].hash;
    if (!ok) {
        skip[i] = 1;
        set_status(c.status, SAE_ST_BAD_BLOCK);
        return;
    }
    if (SAE_HASH_RESERVED(h)) {
        skip[i] = 1;
        set_status(c.status, SAE_ST_BAD_HASH);
        return;
    }
    if (mg & SAE_META_VALID) {
        skip[i] = 1;
        set_status(c.status, SAE_ST_SLOT_BUSY);
        return;
    }
    skip[i] = 0;
    uint32_t m = meta[i] & (0x7u | (0x7u << 3) | (0xFu << 9));
    c.meta[g] = (uint16_t)(m | SAE_META_VALID | SAE_META_LEAF);
    c.la[g] = la[i];
    c.off[g] = off[i];
    c.hash[g] = h;
    c.parent[g] = parent[i];
    c.child_count[g] = 0;
    c.ref_count[g] = 0;
    c.access_count[g] = 0;
    if (!index_insert_from(tab, c.index_mask, h, b, slot_tq(m, off[i]), si, vi))
        set_status(c.status, SAE_ST_INDEX_FULL);
    int32_t *cs = counter_slot(c, inst, i);
    atomicAdd(cs + SAE_CF_RES + meta_queue(m), 1);
    if (c.state[inst].learn & SAE_LEARN_TOKEN_EMA) atomicAdd(cs + SAE_CF_TADD + meta_type(m) % SAE_N_TYPES, 1);
    // recently_evicted: a hit counts one miss after eviction (Algorithm 1,
    // Add) and consumes the entry; its table slot then stays stale (a lookup
    // skips a consumed entry) until the table is rebuilt from the ring
    uint32_t rp = 0;
    if (ghost_find_from(gt, c.ghost_mask, ring, h, c.state[inst].ev_count, c.W, sg, vg, &rp) >= 0) {
        const uint32_t old = atomicOr(&ring[rp].tq, SAE_TQ_CONSUMED);
        if (!(old & SAE_TQ_CONSUMED)) {
            atomicAdd(cs + SAE_CF_MISSED + (old & 7u) % SAE_N_TYPES, 1);
            if (((c.struct_mask >> ((old >> 3) & 7u)) & 1u) && (c.state[inst].learn & SAE_LEARN_DECAY_POWER))
                atomicAdd(cs + SAE_CF_BMISS + ((old >> SAE_TQ_BIN_SHIFT) & (SAE_N_BINS - 1)), 1);
        }
    }
}

// Add(), phase 2: parents gain a child and stop being leaves.
__global__ void k_insert_b(DevCtx c, int n, const int32_t *inst_a, const int32_t *parent, const uint8_t *skip)
{
    int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n || skip[i]) return;
    int inst = inst_a ? inst_a[i] : 0;
    int32_t p = parent[i];
    if (p < 0) return;
    if (p >= c.N) {
        set_status(c.status, SAE_ST_BAD_BLOCK);
        return;
    }
    long long gp = (long long)inst * c.N + p;
    atomicAdd(&c.child_count[gp], 1);
    meta_and(c.meta, gp, (uint32_t)(~SAE_META_LEAF) & 0xFFFFu);
}

__global__ void k_ref_a(DevCtx c, int n, const int32_t *inst_a, const int32_t *ids, int32_t delta)
{
    int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    int inst = inst_a ? inst_a[i] : 0;
    int32_t b = ids[i];
    if (inst < 0 || inst >= c.n_inst || b < 0 || b >= c.N) {
        set_status(c.status, SAE_ST_BAD_BLOCK);
        return;
    }
    atomicAdd(&c.ref_count[(long long)inst * c.N + b], delta);
}
__global__ void k_ref_b(DevCtx c, int n, const int32_t *inst_a, const int32_t *ids)
{
    int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    int inst = inst_a ? inst_a[i] : 0;
    int32_t b = ids[i];
    if (inst < 0 || inst >= c.n_inst || b < 0 || b >= c.N) return;
    long long g = (long long)inst * c.N + b;
    if (c.ref_count[g] > 0) meta_or(c.meta, g, SAE_META_REF);
    else meta_and(c.meta, g, (uint32_t)(~SAE_META_REF) & 0xFFFFu);
}

// One wave per request, kThreads per workgroup (prefix_match_wg).
__global__ void __launch_bounds__(kThreads) k_prefix_match(DevCtx c, PmArgs pa)
{
    __shared__ PmShared<kThreads> sh;
    prefix_match_wg<kThreads>(c, blockIdx.x, pa, sh);
}


// Second pass of a prefix match with SAE_PM_INTERVALS, 1024 threads per
// workgroup.  Workgroups 0 .. n_inst-1 append instance i's intervals to its
// rings in request order: each round gives thread t the PLACE_R requests
// t*PLACE_R .. t*PLACE_R+PLACE_R-1 of the round (one round trip for all of
// their records), a workgroup scan per log-normal queue ranks them, and a
// later round overwrites the ring slots of an earlier one in rank order (the
// barrier between rounds orders the stores).  The other workgroups touch every
// matched block (SAE_PM_TOUCH).  Neither part reads what the other writes.
constexpr int kPlaceThreads = 1024;
constexpr int PLACE_R = 4;
__global__ void __launch_bounds__(kPlaceThreads) k_pm_place(DevCtx c, int n_req, int max_len, const int32_t *inst_a,
                                                           int32_t now, uint32_t flags, const int32_t *matched_ids)
{
    constexpr int NW = kPlaceThreads / SAE_WAVE;
    __shared__ uint32_t wsum[NW];
    const int lane = (int)__lane_id();
    const int wave = threadIdx.x / SAE_WAVE;
    if ((int)blockIdx.x >= c.n_inst) {
        if (!(flags & SAE_PM_TOUCH)) return;
        const long long total = (long long)n_req * max_len;
        const long long stride = (long long)(gridDim.x - c.n_inst) * kPlaceThreads;
        for (long long e = (long long)(blockIdx.x - c.n_inst) * kPlaceThreads + threadIdx.x; e < total; e += stride) {
            const int32_t id = matched_ids[e];
            if (id < 0) continue;
            const int r = (int)(e / max_len);
            const int inst = inst_a ? inst_a[r] : 0;
            const long long g = (long long)inst * c.N + id;
            c.la[g] = now;
            atomicAdd(&c.access_count[g], 1);
        }
        return;
    }
    const int i = blockIdx.x;
    InstState &s = c.state[i];
    long long n0[SAE_MAX_QUEUES];
#pragma unroll
    for (int q = 0; q < SAE_MAX_QUEUES; ++q) n0[q] = ((c.ln_mask >> q) & 1u) ? s.ivl_n[q] : 0;
    long long run[SAE_MAX_QUEUES];
#pragma unroll
    for (int q = 0; q < SAE_MAX_QUEUES; ++q) run[q] = 0;
    for (int base = 0; base < n_req; base += kPlaceThreads * PLACE_R) {
        const int r0 = base + threadIdx.x * PLACE_R;
        // every load is issued unconditionally (a clamped index) and masked
        // afterwards, so the loads of all PLACE_R requests are in flight together
        int32_t v[PLACE_R][SAE_MAX_QUEUES];  // dt per request and queue; 0: none
#pragma unroll
        for (int u = 0; u < PLACE_R; ++u) {
            const int r = r0 + u;
            const int rc = r < n_req ? r : n_req - 1;
            const int ri = inst_a ? inst_a[rc] : 0;
            const bool mine = r < n_req && ri == i;
            const int4 *src = reinterpret_cast<const int4 *>(c.pm_rec + (long long)rc * SAE_MAX_QUEUES);
            const int4 a = src[0], b = src[1];
            v[u][0] = mine ? a.x : 0; v[u][1] = mine ? a.y : 0; v[u][2] = mine ? a.z : 0; v[u][3] = mine ? a.w : 0;
            v[u][4] = mine ? b.x : 0; v[u][5] = mine ? b.y : 0; v[u][6] = mine ? b.z : 0; v[u][7] = mine ? b.w : 0;
        }
#pragma unroll
        for (int q = 0; q < SAE_MAX_QUEUES; ++q) {
            if (!((c.ln_mask >> q) & 1u)) continue;
            uint32_t mine = 0;
#pragma unroll
            for (int u = 0; u < PLACE_R; ++u) mine += v[u][q] > 0 ? 1u : 0u;
            // inclusive scan over the wave, then over the waves
            uint32_t inc = mine;
#pragma unroll
            for (int o = 1; o < SAE_WAVE; o <<= 1) {
                const uint32_t t = __shfl_up(inc, o);
                if (lane >= o) inc += t;
            }
            __syncthreads();  // wsum of the previous scan has been read
            if (lane == SAE_WAVE - 1) wsum[wave] = inc;
            __syncthreads();
            uint32_t before = 0, round_total = 0;
#pragma unroll
            for (int w = 0; w < NW; ++w) {
                const uint32_t x = wsum[w];
                before += (w < wave) ? x : 0u;
                round_total += x;
            }
            long long rank = run[q] + before + (inc - mine);
            int32_t *ring = c.ivl + ((long long)i * c.Q + q) * SAE_IVL_CAP;
#pragma unroll
            for (int u = 0; u < PLACE_R; ++u) {
                if (v[u][q] > 0) {
                    ring[(n0[q] + rank) % SAE_IVL_CAP] = v[u][q];
                    ++rank;
                }
            }
            run[q] += round_total;
        }
        __syncthreads();  // this round's ring stores precede the next round's
    }
    if (threadIdx.x == 0) {
#pragma unroll
        for (int q = 0; q < SAE_MAX_QUEUES; ++q)
            if ((c.ln_mask >> q) & 1u) s.ivl_n[q] = n0[q] + run[q];
    }
}

// ---------------------------------------------------------------------------
// Commit, per victim: free the block, erase its index entry, count it
// (Algorithm 3 evicted[tau], Algorithm 2 queue_evictions[q]), update its
// parent and record it in recently_evicted.
constexpr int kCommitThreads = 64;
static_assert(SAE_CF_N <= kCommitThreads, "one thread per counter field");
__global__ void __launch_bounds__(kCommitThreads) k_commit(DevCtx c, const int32_t *decision)
{
    __shared__ int32_t sums[SAE_CF_N];
    const int inst = blockIdx.y;
    const int j = blockIdx.x * blockDim.x + threadIdx.x;
    if (threadIdx.x < SAE_CF_N) sums[threadIdx.x] = 0;
    __syncthreads();
    const InstState &s = c.state[inst];
    // the decision entry is loaded with the decision size (j < max_k: in
    // bounds either way), so that both arrive in one round trip
    const int32_t vj = decision[(long long)inst * c.max_k + (j < c.max_k ? j : 0)];
    const int d = s.last_d;
    int32_t v = (j < d) ? vj : -1;
    if (j < d && (v < 0 || v >= c.N)) {
        set_status(c.status, SAE_ST_BAD_BLOCK);
        v = -1;
    }
    if (v >= 0) commit_victim(c, inst, j, v, s.ev_before, d, sums);
    __syncthreads();
    if (threadIdx.x < SAE_CF_N && sums[threadIdx.x])
        atomicAdd(counter_slot(c, inst, blockIdx.x) + threadIdx.x, sums[threadIdx.x]);
}

inline unsigned grid_for(long long n) { return (unsigned)((n + kThreads - 1) / kThreads); }

// The recipe's elementary functions, element-wise (sae_recipe_eval).
__global__ void k_recipe_eval(int fn, long long n, const float *x, float *y)
{
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x) {
        const float v = x[i];
        y[i] = (fn == SAE_FN_LN) ? dsr::ln(v) : ((fn == SAE_FN_EXP) ? dsr::exp(v) : dsr::erfc(v));
    }
}

}  // namespace

hipError_t launch_recipe_eval(int fn, int64_t n, const float *x, float *y, hipStream_t s)
{
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_recipe_eval, dim3(grid_for(n)), dim3(kThreads), 0, s, fn, (long long)n, x, y);
    return hipGetLastError();
}

hipError_t launch_block_type(const uint8_t *counts, int64_t n, uint8_t *tau, hipStream_t s)
{
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_block_type, dim3(grid_for(n)), dim3(kThreads), 0, s, counts, (long long)n, tau);
    return hipGetLastError();
}

hipError_t launch_classify(int n, const uint8_t *hint, uint16_t *meta, const int32_t *roles, hipStream_t s)
{
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_classify, dim3(grid_for(n)), dim3(kThreads), 0, s, n, hint, meta, roles[0], roles[1],
                       roles[2], roles[3]);
    return hipGetLastError();
}

hipError_t launch_index_build(const DevCtx &c, hipStream_t s)
{
    long long nidx = (long long)c.n_inst * ((long long)c.index_mask + 1);
    long long ngt = (long long)c.n_inst * ((long long)c.ghost_mask + 1);
    long long nring = (long long)c.n_inst * c.ring_cap;
    long long n = nidx;
    if (ngt > n) n = ngt;
    if (nring > n) n = nring;
    if (c.n_inst > n) n = c.n_inst;
    if ((long long)c.n_inst * SAE_CSLOTS * SAE_CF_STRIDE > n) n = (long long)c.n_inst * SAE_CSLOTS * SAE_CF_STRIDE;
    hipLaunchKernelGGL(k_clear_all, dim3(grid_for(n)), dim3(kThreads), 0, s, c, 1);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_index_fill, dim3(grid_for((long long)c.n_inst * c.N)), dim3(kThreads), 0, s, c, 1);
    return hipGetLastError();
}

hipError_t launch_index_rebuild(const DevCtx &c, hipStream_t s)
{
    long long nidx = (long long)c.n_inst * ((long long)c.index_mask + 1);
    hipLaunchKernelGGL(k_clear_all, dim3(grid_for(nidx)), dim3(kThreads), 0, s, c, 0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_index_fill, dim3(grid_for((long long)c.n_inst * c.N)), dim3(kThreads), 0, s, c, 0);
    return hipGetLastError();
}

hipError_t launch_ghost_rebuild(const DevCtx &c, hipStream_t s)
{
    long long ngt = (long long)c.n_inst * ((long long)c.ghost_mask + 1);
    hipLaunchKernelGGL(k_ghost_clear, dim3(grid_for(ngt)), dim3(kThreads), 0, s, c);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    long long nring = (long long)c.n_inst * c.ring_cap;
    hipLaunchKernelGGL(k_ghost_fill, dim3(grid_for(nring)), dim3(kThreads), 0, s, c);
    return hipGetLastError();
}

hipError_t launch_insert(const DevCtx &c, int32_t n, const int32_t *inst, const int32_t *ids, const uint64_t *hash,
                         const int32_t *parent, const int32_t *la, const uint16_t *meta, const uint32_t *off,
                         uint8_t *skip, hipStream_t s)
{
    if (n <= 0) return hipSuccess;
    // one wave per workgroup: an insert is a chain of scattered accesses, so
    // the inserts are spread over as many compute units as possible
    const unsigned grid = (unsigned)(((long long)n + kCommitThreads - 1) / kCommitThreads);
    hipLaunchKernelGGL(k_insert_a, dim3(grid), dim3(kCommitThreads), 0, s, c, n, inst, ids, hash, parent, la, meta,
                       off, skip);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_insert_b, dim3(grid), dim3(kCommitThreads), 0, s, c, n, inst, parent, (const uint8_t *)skip);
    return hipGetLastError();
}

hipError_t launch_ref(const DevCtx &c, int32_t n, const int32_t *inst, const int32_t *ids, int32_t delta, hipStream_t s)
{
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_ref_a, dim3(grid_for(n)), dim3(kThreads), 0, s, c, n, inst, ids, delta);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_ref_b, dim3(grid_for(n)), dim3(kThreads), 0, s, c, n, inst, ids);
    return hipGetLastError();
}

hipError_t launch_pm_place(const DevCtx &c, int32_t n_req, int32_t max_len, const int32_t *inst, int32_t now,
                           uint32_t flags, const int32_t *matched_ids, hipStream_t s)
{
    long long tg = 0;
    if (flags & SAE_PM_TOUCH) tg = ((long long)n_req * max_len + kPlaceThreads - 1) / kPlaceThreads;
    if (tg > 1024) tg = 1024;
    hipLaunchKernelGGL(k_pm_place, dim3((unsigned)(c.n_inst + tg)), dim3(kPlaceThreads), 0, s, c, n_req, max_len,
                       inst, now, flags, matched_ids);
    return hipGetLastError();
}

hipError_t launch_prefix_match(const DevCtx &c, int32_t n_req, int32_t max_len, const uint64_t *hashes,
                               const int32_t *lens, const int32_t *inst, int32_t now, uint32_t flags,
                               int32_t *match_len, int32_t *matched_ids, hipStream_t s)
{
    if (n_req <= 0) return hipSuccess;
    const long long threads = (long long)n_req * SAE_WAVE;
    const PmArgs pa = {n_req, max_len, hashes, lens, inst, now, flags, match_len, matched_ids};
    hipLaunchKernelGGL(k_prefix_match, dim3(grid_for(threads)), dim3(kThreads), 0, s, c, pa);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !(flags & SAE_PM_INTERVALS)) return e;
    return launch_pm_place(c, n_req, max_len, inst, now, flags, matched_ids, s);
}

hipError_t launch_commit(const DevCtx &c, const SelectArgs &a, hipStream_t s)
{
    // one wave per workgroup: a victim is a chain of scattered accesses, so
    // the victims are spread over as many compute units as possible
    dim3 grid((unsigned)((c.max_k + kCommitThreads - 1) / kCommitThreads), (unsigned)c.n_inst);
    hipLaunchKernelGGL(k_commit, grid, dim3(kCommitThreads), 0, s, c, (const int32_t *)a.decision);
    return hipGetLastError();
}
