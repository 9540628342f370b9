// Internal definitions shared by the HIP translation units of libsae.
// Target: gfx950 (CDNA4), wave64.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sae.h"

#define SAE_WAVE 64
#define SAE_EMPTY_HASH 0ull
#define SAE_TOMB_HASH 0xFFFFFFFFFFFFFFFFull
// The two reserved hash values mark empty and deleted table slots: a block
// carrying one is never indexed, never found and never recorded as evicted.
#define SAE_HASH_RESERVED(h) ((h) == SAE_EMPTY_HASH || (h) == SAE_TOMB_HASH)
#define SAE_MAX_PROBES 65536

// Radix digits of the selection: 11 bits -> 2048 bins.
#define SAE_DIGIT_BITS 11
#define SAE_BINS (1 << SAE_DIGIT_BITS)

// Sampling of the pool-scan engine: chunks per instance and blocks per chunk.
#define SAE_SAMPLE_WGS 64
#define SAE_SAMPLE_CHUNK 256
// Candidate buckets of the pool-scan engine, per (instance, queue): the bucket
// upper ends are sampled (key, id) values at or below the candidate bound.
#define SAE_NBUCKET 256  // buckets
#define SAE_LCAP 16384   // candidates kept per (instance, queue)
// The scan appends a queue's candidates to one of SAE_STRIPES stripes of
// SAE_LCAP / SAE_STRIPES slots (one device atomic per workgroup and queue,
// spread over the stripes so that few workgroups meet on one counter); what
// does not fit a stripe goes to the queue's overflow list of SAE_LCAP slots.
#define SAE_STRIPES 64
#define SAE_STRIPE_CAP (SAE_LCAP / SAE_STRIPES)

// Feedback counters are added into one of SAE_CSLOTS striped copies (chosen by
// the adding workgroup) and folded into InstState by the learner kernel:
// device-wide atomics on one address serialise, so many workgroups must not
// add into the same word.
#define SAE_CSLOTS 64
#define SAE_CF_EVICTED 0     // 5 fields, token_stats[tau].evicted
#define SAE_CF_MISSED 5      // 5 fields, token_stats[tau].miss_after_evict
#define SAE_CF_HITS 10       // 8 fields, queue_hits[q]
#define SAE_CF_EVICTIONS 18  // 8 fields, queue_evictions[q]
#define SAE_CF_BHITS 26      // 8 fields, hits of structural blocks per positional bin
#define SAE_CF_BMISS 34      // 8 fields, misses after eviction per positional bin
#define SAE_CF_THITS 42      // 5 fields, prefix-match hits per block type
#define SAE_CF_TADD 47       // 5 fields, blocks added per type
#define SAE_CF_RES 52        // 8 fields, change of the cached blocks per queue
#define SAE_CF_N 60
#define SAE_CF_STRIDE 64

// recently_evicted entry bits: tau | queue << 3 | consumed | positional bin << 9
#define SAE_TQ_CONSUMED 0x100u
#define SAE_TQ_BIN_SHIFT 9

// ----------------------------------------------------------------------------
// Per-instance device state: learned parameters, learner settings and the
// feedback counters of Algorithms 1-3.
struct InstState {
    float w[SAE_N_TYPES];
    float alpha[SAE_MAX_QUEUES];
    float mu[SAE_MAX_QUEUES];
    float sigma[SAE_MAX_QUEUES];
    float gamma, eta, T, beta, beta_ln;
    int32_t K;
    uint32_t learn;
    int32_t evicted[SAE_N_TYPES];
    int32_t missed[SAE_N_TYPES];
    int32_t hits[SAE_MAX_QUEUES];
    int32_t evictions[SAE_MAX_QUEUES];
    long long ev_count;   // evictions so far
    long long ev_before;  // ev_count before the last committed decision
    int32_t pending;      // learners due
    int32_t n_updates;
    int32_t last_d;       // size of the last committed decision
    int32_t bin_hits[SAE_N_BINS];    // decay-power learner counters
    int32_t bin_missed[SAE_N_BINS];
    int32_t type_hits[SAE_N_TYPES];  // text-form token-weight counters
    int32_t type_added[SAE_N_TYPES];
    int32_t resident[SAE_MAX_QUEUES];  // cached blocks per queue
    long long ivl_n[SAE_MAX_QUEUES];      // Algorithm 4: intervals recorded so far, per queue
    long long ivl_start[SAE_MAX_QUEUES];  // first interval still in the buffer (before the cap)
};

// Open-addressing slot of the block index: content hash -> block id, with the
// block's type, queue and positional bin as of its insertion (the layout of
// GhostEntry.tq without the consumed bit), so a prefix match counts its hits
// without reading the pool.
struct IndexSlot {
    unsigned long long hash;  // SAE_EMPTY_HASH, SAE_TOMB_HASH or a content hash
    int32_t id;
    uint32_t tq;  // tau | queue << 3 | pos_bin << SAE_TQ_BIN_SHIFT
};

// recently_evicted: a ring in eviction order plus a hash table into it.
struct GhostEntry {
    unsigned long long hash;  // 0 when the ring slot was never written
    long long stamp;          // eviction_count right after the entry's decision
    uint32_t tq;              // tau | queue << 3 | consumed << 8
    uint32_t pad_;
};
struct GhostSlot {
    unsigned long long hash;
    uint32_t ring;  // ring position of the entry
    uint32_t pad_;
};

// Everything a kernel needs about a context, passed by value.
struct DevCtx {
    int32_t n_inst, N, Q, max_k;
    int32_t kind[SAE_MAX_QUEUES];
    int32_t ef_queue;  // index of the evict-first queue or -1
    int32_t W;         // ghost window
    int32_t ring_cap;  // W + max_k
    uint32_t index_mask, ghost_mask;
    // pool (caller-owned)
    int32_t *la;
    uint16_t *meta;
    uint32_t *off;
    unsigned long long *hash;
    int32_t *parent;
    int32_t *child_count;
    int32_t *ref_count;
    int32_t *access_count;
    // context-owned
    InstState *state;
    uint32_t *status;
    IndexSlot *index;     // [n_inst][index_mask + 1]
    GhostEntry *ring;     // [n_inst][ring_cap]
    GhostSlot *gtab;      // [n_inst][ghost_mask + 1]
    unsigned long long *thr;   // [n_inst][Q] candidate bound on (key << 32 | id), scan engine
    uint4 *sent;               // [n_inst][64] scan filter entry of each (type, queue), index type << 3 | queue
    int32_t *eflim;            // [n_inst][16] evict-first queue: largest candidate id per num_tokens - 1 (-1: none)
    unsigned long long *samp;  // [n_inst][SAE_SAMPLE_WGS][SAE_SAMPLE_CHUNK] sampled (key << 32 | id)
    uint32_t *samp_qn;         // [n_inst][SAE_SAMPLE_WGS][SAE_MAX_QUEUES] sampled elements per chunk and queue
    uint32_t *prep_done;       // [n_inst] sampling workgroups of sae_match_select finished, ever (wraps)
    uint32_t *sel_stats;       // [n_inst][Q][4] last pool scan: evictable, candidates, beyond a stripe, slow path
    unsigned long long *split; // [n_inst][Q][SAE_NBUCKET] bucket upper ends, ascending; the last is thr
    int32_t *nsplit;           // [n_inst][Q] buckets (0: no candidates)
    unsigned long long *cand;  // [n_inst][Q][2 SAE_LCAP] candidates, unordered: the stripes
                               // (SAE_STRIPES x SAE_STRIPE_CAP), then the overflow list
    uint32_t *stripe_n;        // [n_inst][Q][SAE_STRIPES + 1] slots taken in each stripe (may exceed its
                               // capacity: the rest went to the overflow list), then in the overflow list
    int32_t scan_gx;           // scan workgroups per instance
    int32_t n_cu;              // compute units of the device
    int32_t *cpart;            // [n_inst][SAE_CSLOTS][SAE_CF_STRIDE] feedback counters, striped
    unsigned long long *sel;   // [n_inst][Q][max_k]   sorted selection
    int32_t *sel_count;        // [n_inst][Q]
    int32_t *ivl;              // [n_inst][Q][SAE_IVL_CAP] Algorithm 4 interval rings (dt in ticks)
    int32_t *pm_rec;           // [max_requests][SAE_MAX_QUEUES] intervals of one prefix-match call (0: none)
    int32_t max_req;
    uint32_t ln_mask;          // bit q: queue q is log-normal
    uint32_t struct_mask;      // bit q: queue q is structural
    // cascading decisions (SAE_SS_CASCADE): per block, cached children found
    // among the candidates so far and the largest rank among them, and the
    // blocks whose entries a call changed with their count.  Two sets that
    // calls alternate between: a call's first round clears what the previous
    // call left in the other set (the pointers below are the call's own set
    // and, in the *_prev fields, the other one).
    int32_t *casc_cnt;              // [n_inst][N]
    unsigned long long *casc_e;     // [n_inst][N]
    int32_t *casc_touch;            // [n_inst][casc_tl]
    int32_t *casc_nt;               // [n_inst] touched blocks of the set's last call
    int32_t *casc_cnt_prev;
    unsigned long long *casc_e_prev;
    int32_t *casc_touch_prev;
    int32_t *casc_nt_prev;
    int32_t casc_tl;
    // the first round's output: kappa of each snapshot victim, the parents
    // whose last cached child it was, those of them below the admission
    // bound with their E, and per instance the counts of touched blocks,
    // listed and admitted parents (zero between calls) and the call's final
    // count of touched blocks
    unsigned long long *casc_k0;    // [n_inst][max_k]
    int32_t *casc_prom;             // [n_inst][max_k]
    int32_t *casc_aid;              // [n_inst][max_k]
    unsigned long long *casc_pe;    // [n_inst][max_k]
    int32_t *casc_n;                // [n_inst][4]: touched, listed, (unused), admitted
    // Batched engine (instances of at most 65,536 blocks): every block's key
    // and queue + 1 (0: not evictable) from the call's first pass, read back
    // by its later passes
    uint32_t *bkey;  // [n_inst][N]
    uint8_t *bq;     // [n_inst][N]
};

// Positional bin of a block (decay-power learner): floor(8 o_b / o_max) with
// o_b capped at o_max, 7 at the end, 0 for a one-block template (o_max = 0).
__device__ __forceinline__ uint32_t pos_bin(uint32_t off)
{
    const uint32_t ob = off & 0xFFFFu, omax = off >> 16;
    if (omax == 0) return 0;
    const uint32_t b = (SAE_N_BINS * (ob < omax ? ob : omax)) / omax;
    return b < SAE_N_BINS - 1 ? b : SAE_N_BINS - 1;
}

// ----------------------------------------------------------------------------
// Meta field access.
__device__ __forceinline__ int meta_queue(uint32_t m) { return (int)(m & 7u); }
__device__ __forceinline__ int meta_type(uint32_t m) { return (int)((m >> 3) & 7u); }

// Type, queue and positional bin of a block (meta m, offsets off) packed as
// tau | queue << 3 | pos_bin << SAE_TQ_BIN_SHIFT: the recently_evicted entry
// and the index slot of the block carry it.
__device__ __forceinline__ uint32_t slot_tq(uint32_t m, uint32_t off)
{
    return (uint32_t)(meta_type(m) % SAE_N_TYPES) | ((uint32_t)meta_queue(m) << 3) |
           (pos_bin(off) << SAE_TQ_BIN_SHIFT);
}
__device__ __forceinline__ int meta_ntok(uint32_t m) { return (int)((m >> 9) & 15u) + 1; }
__device__ __forceinline__ bool meta_evictable(uint32_t m)
{
    return (m & (SAE_META_VALID | SAE_META_LEAF | SAE_META_REF)) == (SAE_META_VALID | SAE_META_LEAF);
}

// 32-bit atomics on the 16-bit meta of block `b` (meta base is 4-byte aligned).
__device__ __forceinline__ void meta_and(uint16_t *meta, long long b, uint32_t mask16)
{
    uint32_t *w = reinterpret_cast<uint32_t *>(meta + (b & ~1ll));
    uint32_t sh = (uint32_t)(b & 1) * 16u;
    atomicAnd(w, ~((~mask16 & 0xFFFFu) << sh));
}
__device__ __forceinline__ void meta_or(uint16_t *meta, long long b, uint32_t bits16)
{
    uint32_t *w = reinterpret_cast<uint32_t *>(meta + (b & ~1ll));
    uint32_t sh = (uint32_t)(b & 1) * 16u;
    atomicOr(w, (bits16 & 0xFFFFu) << sh);
}

__device__ __forceinline__ int32_t *counter_slot(const DevCtx &c, int inst, int slot)
{
    return c.cpart + ((long long)inst * SAE_CSLOTS + (slot & (SAE_CSLOTS - 1))) * SAE_CF_STRIDE;
}

__device__ __forceinline__ void set_status(uint32_t *status, uint32_t bits)
{
    if (bits) atomicOr(status, bits);
}

// Hash -> home slot.
__device__ __forceinline__ uint32_t hash_home(unsigned long long h, uint32_t mask)
{
    unsigned long long z = h ^ (h >> 31);
    z *= 0x9E3779B97F4A7C15ull;
    return (uint32_t)(z >> 32) & mask;
}

// index_erase and ghost_insert continued from the home slot s0 whose hash v0
// the caller has already loaded (so that several first probes can be in
// flight together): linear probing from the home slot, as every lookup of
// the block index and of recently_evicted does.
__device__ __forceinline__ void index_erase_from(IndexSlot *tab, uint32_t mask, unsigned long long h, uint32_t s0,
                                                 unsigned long long v0)
{
    uint32_t s = s0;
    unsigned long long v = v0;
    for (int p = 0; p <= (int)mask && p < SAE_MAX_PROBES; ++p) {
        if (p > 0) v = tab[s].hash;
        if (v == h) {
            tab[s].hash = SAE_TOMB_HASH;
            return;
        }
        if (v == SAE_EMPTY_HASH) return;
        s = (s + 1) & mask;
    }
}

__device__ __forceinline__ bool ghost_insert_from(GhostSlot *tab, uint32_t mask, unsigned long long h,
                                                  uint32_t ring_pos, uint32_t s0, unsigned long long v0)
{
    uint32_t s = s0;
    unsigned long long v = v0;
    bool fresh = true;  // v holds slot s's hash as loaded
    for (int p = 0; p <= (int)mask && p < SAE_MAX_PROBES; ++p) {
        if (!fresh) v = tab[s].hash;
        fresh = false;
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

// Commit of victim v at decision position j (of d) of instance inst: free the
// block, erase its index entry, count it into the LDS sums (Algorithm 3's
// evicted[tau], Algorithm 2's queue_evictions[q], the queue's cached
// blocks), take it from its parent (a parent left without a cached child
// becomes a leaf) and record it in recently_evicted at ring position
// evb + j, stamped evb + d (evb: eviction_count before the decision).
__device__ __forceinline__ void commit_victim(const DevCtx &c, int inst, int j, int32_t v, long long evb, int d,
                                              int32_t *sums)
{
    const long long g = (long long)inst * c.N + v;
    // one round trip for the block's fields, then one for the parent's
    // count and the first probes of both tables together
    const uint32_t m = c.meta[g];
    const unsigned long long h = c.hash[g];
    const int32_t p = c.parent[g];
    const uint32_t off = c.off[g];
    IndexSlot *tab = c.index + (long long)inst * ((long long)c.index_mask + 1);
    GhostSlot *gt = c.gtab + (long long)inst * ((long long)c.ghost_mask + 1);
    const uint32_t si = hash_home(h, c.index_mask), sg = hash_home(h, c.ghost_mask);
    const unsigned long long vi = tab[si].hash, vg = gt[sg].hash;
    const bool has_p = p >= 0 && p < c.N;
    const long long gp = (long long)inst * c.N + (has_p ? p : 0);
    const int before = has_p ? atomicSub(&c.child_count[gp], 1) : 0;
    atomicAdd(&sums[SAE_CF_EVICTED + meta_type(m) % SAE_N_TYPES], 1);
    atomicAdd(&sums[SAE_CF_EVICTIONS + meta_queue(m)], 1);
    atomicSub(&sums[SAE_CF_RES + meta_queue(m)], 1);
    meta_and(c.meta, g, (uint32_t)(~SAE_META_VALID) & 0xFFFFu);
    const bool hashed = !SAE_HASH_RESERVED(h);  // a reserved hash was never indexed
    if (hashed) index_erase_from(tab, c.index_mask, h, si, vi);
    if (has_p && before == 1) meta_or(c.meta, gp, SAE_META_LEAF);
    GhostEntry *ring = c.ring + (long long)inst * c.ring_cap;
    const uint32_t rp = (uint32_t)((evb + j) % c.ring_cap);
    GhostEntry e;
    e.hash = hashed ? h : SAE_EMPTY_HASH;  // an empty entry is never found
    e.stamp = evb + d;
    e.tq = slot_tq(m, off);
    e.pad_ = 0;
    ring[rp] = e;
    if (hashed && !ghost_insert_from(gt, c.ghost_mask, h, rp, sg, vg)) set_status(c.status, SAE_ST_GHOST_FULL);
}

// ----------------------------------------------------------------------------
// Deterministic fp32 realisation of Eq. 1-3.  Only IEEE binary32 + - * /,
// fmaf, int<->float conversion and exact bit operations, in a fixed order
// (built with -ffp-contract=off).  The same recipe is evaluated on the CPU by
// the test oracle; both are transcriptions of one specification, so the
// selection -- an argmin decided in fp32 -- comes out identical.
//   ln:   x = 2^e m, m in (sqrt(1/2), sqrt(2)]; ln m = 2 atanh(s), s = (m-1)/(m+1),
//         atanh series through s^9/9; ln 2 = head (15 bits) + tail (Cody-Waite).
//   exp:  n = rint(y / ln 2), r = y - n ln 2 (head, then tail), Taylor series of
//         e^r through r^7/7!, times 2^n built in the exponent field;
//         0 below y = -86, +inf above 88.
//   erfc: x >= 0: t exp(-x^2 + g(t)), t = 1/(1 + x/2), g of degree 9 with the
//         Chebyshev-fitted coefficients of Press et al., Numerical Recipes
//         (2nd ed., Sec. 6.2); x^2 kept as an exact head + tail.
//         erfc(0) = 1, erfc(x >= 9) = 0.
namespace dsr {

__device__ __forceinline__ float pow2i(int n) { return __uint_as_float((uint32_t)(n + 127) << 23); }

// e^r, |r| <= ~0.35
__device__ __forceinline__ float exp_series(float r)
{
    float p = 1.0f / 5040.0f;
    p = fmaf(p, r, 1.0f / 720.0f);
    p = fmaf(p, r, 1.0f / 120.0f);
    p = fmaf(p, r, 1.0f / 24.0f);
    p = fmaf(p, r, 1.0f / 6.0f);
    p = fmaf(p, r, 0.5f);
    p = fmaf(p, r, 1.0f);
    p = fmaf(p, r, 1.0f);
    return p;
}

constexpr float kLn2Hi = 0x1.62e400p-1f;
constexpr float kLn2Lo = 0x1.7f7d1cp-20f;
constexpr float kInvLn2 = 0x1.715476p+0f;
constexpr float kRound = 0x1.8p+23f;
constexpr float kSqrt2 = 0x1.6a09e6p+0f;

// Branch-free: the arithmetic runs on y clamped into [-86, 88]; results
// outside are then replaced (identical values for every finite y).
__device__ __forceinline__ float exp(float y)
{
    const float yc = fminf(fmaxf(y, -86.0f), 88.0f);
    const float n = (yc * kInvLn2 + kRound) - kRound;
    float r = fmaf(-n, kLn2Hi, yc);
    r = fmaf(-n, kLn2Lo, r);
    float v = exp_series(r) * pow2i((int)n);
    v = (y < -86.0f) ? 0.0f : v;
    v = (y > 88.0f) ? __uint_as_float(0x7F800000u) : v;
    return v;
}

__device__ __forceinline__ float ln(float x)
{
    uint32_t bits = __float_as_uint(x);
    int e = (int)(bits >> 23) - 127;
    uint32_t mb = (bits & 0x007FFFFFu) | 0x3F800000u;
    if (mb > 0x3FB504F3u) {
        mb -= 0x00800000u;
        e += 1;
    }
    float f = __uint_as_float(mb) - 1.0f;
    float s = f / (2.0f + f);
    float z = s * s;
    float q = fmaf(z, 1.0f / 9.0f, 1.0f / 7.0f);
    q = fmaf(z, q, 1.0f / 5.0f);
    q = fmaf(z, q, 1.0f / 3.0f);
    float s2 = s + s;
    float lnm = fmaf(s2 * z, q, s2);
    float ef = (float)e;
    return fmaf(ef, kLn2Hi, fmaf(ef, kLn2Lo, lnm));
}

// x >= 0.  Branch-free: the arithmetic runs on min(x, 9); erfc(0) = 1 and
// erfc(x >= 9) = 0 are selected afterwards.
__device__ __forceinline__ float erfc(float x)
{
    const float xc = fminf(x, 9.0f);
    const float t = 1.0f / fmaf(0.5f, xc, 1.0f);
    float g = 0.17087277f;
    g = fmaf(g, t, -0.82215223f);
    g = fmaf(g, t, 1.48851587f);
    g = fmaf(g, t, -1.13520398f);
    g = fmaf(g, t, 0.27886807f);
    g = fmaf(g, t, -0.18628806f);
    g = fmaf(g, t, 0.09678418f);
    g = fmaf(g, t, 0.37409196f);
    g = fmaf(g, t, 1.00002368f);
    g = fmaf(g, t, -1.26551223f);
    const float xx = xc * xc;
    const float xxl = fmaf(xc, xc, -xx);
    const float n = ((g - xx) * kInvLn2 + kRound) - kRound;
    float r = fmaf(-n, kLn2Hi, -xx);
    r = r + g;
    r = r - xxl;
    r = fmaf(-n, kLn2Lo, r);
    float v = t * (exp_series(r) * pow2i((int)n));
    v = (x == 0.0f) ? 1.0f : v;
    v = (x < 9.0f) ? v : 0.0f;
    return v;
}

}  // namespace dsr

// Algorithm 4's summand of an interval: X = x * 2^24 with x the recipe's ln of
// fl32(dt), dt >= 1.  x is 0 (dt = 1) or at least ln 2, so X is an integer
// (< 2^29) and exact.
__device__ __forceinline__ int32_t ivl_scaled_ln(int32_t dt)
{
    return (int32_t)(dsr::ln((float)dt) * 16777216.0f);
}

// Per-instance scoring constants, staged in LDS by every workgroup.
struct ScoreTab {
    float aw[SAE_MAX_QUEUES][8];  // fl(alpha_q * w_tau)
    float mu[SAE_MAX_QUEUES];
    float c[SAE_MAX_QUEUES];      // fl(1 / fl(sigma_q * sqrt 2))
    int32_t kind[SAE_MAX_QUEUES];
    float gamma;
};

// Threads tid = 0 .. 39 of the caller's group fill the table.
__device__ __forceinline__ void load_score_tab(ScoreTab &t, const InstState &s, const DevCtx &c, int tid)
{
    if (tid < SAE_MAX_QUEUES * 8) {
        int q = tid >> 3, ty = tid & 7;
        t.aw[q][ty] = (ty < SAE_N_TYPES) ? s.alpha[q] * s.w[ty] : 0.0f;
    }
    if (tid < SAE_MAX_QUEUES) {
        t.mu[tid] = s.mu[tid];
        t.c[tid] = 1.0f / (s.sigma[tid] * dsr::kSqrt2);
        t.kind[tid] = c.kind[tid];
    }
    if (tid == 0) t.gamma = s.gamma;
}

__device__ __forceinline__ void load_score_tab(ScoreTab &t, const InstState &s, const DevCtx &c)
{
    load_score_tab(t, s, c, (int)threadIdx.x);
}

// Selection key of one block: IEEE bits of P(b) (Eq. 3), or of (float)
// num_tokens for an evict-first queue (Algorithm 1, stage 1).  P >= +0 always,
// so unsigned order of the bits is the numeric order; +inf sorts last.
// One function per queue kind (the pool scan groups blocks by kind so that a
// wave runs one of them without divergence); block_key dispatches.
__device__ __forceinline__ int32_t block_dt(int32_t now, int32_t la, uint32_t &st)
{
    const int32_t dt = now - la;
    st |= (dt < 0) ? (uint32_t)SAE_ST_FUTURE_ACCESS : 0u;
    return dt < 0 ? 0 : dt;
}

// P bits from n = fl(aw p) and dt; dt = 0 gives +inf.  Branch-free.
__device__ __forceinline__ uint32_t priority_bits(float aw, float p, int32_t dt)
{
    const float nn = aw * p;
    const float d = (float)(dt > 0 ? dt : 1);
    const uint32_t b = __float_as_uint(nn / d);
    return dt == 0 ? 0x7F800000u : b;
}

// Eq. 1: 1 - F_LN(dt) = erfc(u)/2, u = (ln dt - mu) c, c = 1 / (sigma sqrt 2).
// Branch-free; dt = 0 (p unused) is evaluated at dt = 1.
__device__ __forceinline__ uint32_t key_lognormal(int32_t now, int32_t la, uint32_t m, const ScoreTab &t,
                                                  uint32_t &st)
{
    const int q = meta_queue(m);
    const int32_t dt = block_dt(now, la, st);
    const float u = (dsr::ln((float)(dt > 0 ? dt : 1)) - t.mu[q]) * t.c[q];
    const float a = fabsf(u);
    const float h = 0.5f * dsr::erfc(a);
    float p = (u >= 0.0f) ? h : 1.0f - h;
    p = dt > 0 ? p : 1.0f;
    return priority_bits(t.aw[q][meta_type(m)], p, dt);
}

// Eq. 2: 1 - (o_b / o_max)^gamma.  Branch-free except on gamma == 1, which is
// the same for every block.
__device__ __forceinline__ uint32_t key_structural(int32_t now, int32_t la, uint32_t m, uint32_t off,
                                                   const ScoreTab &t, uint32_t &st)
{
    const int q = meta_queue(m);
    const int32_t dt = block_dt(now, la, st);
    const int ob = (int)(off & 0xFFFFu), om = (int)(off >> 16);
    st |= (om != 0 && ob > om) ? (uint32_t)SAE_ST_BAD_OFFSET : 0u;
    const float rq = (float)ob / (float)(om != 0 ? om : 1);
    const float r = (om == 0) ? 0.0f : ((ob >= om) ? 1.0f : rq);
    float pw = r;
    if (t.gamma != 1.0f) {
        const float pg = dsr::exp(t.gamma * dsr::ln(r == 0.0f ? 1.0f : r));
        pw = (r == 0.0f) ? 0.0f : ((r == 1.0f) ? r : pg);
    }
    return priority_bits(t.aw[q][meta_type(m)], 1.0f - pw, dt);
}

// Evict-first (num_tokens) and recency (p = 1) queues.
__device__ __forceinline__ uint32_t key_cheap(int kind, int32_t now, int32_t la, uint32_t m, const ScoreTab &t,
                                              uint32_t &st)
{
    const int32_t dt = block_dt(now, la, st);
    const uint32_t rec = priority_bits(t.aw[meta_queue(m)][meta_type(m)], 1.0f, dt);
    return kind == SAE_KIND_EVICT_FIRST ? __float_as_uint((float)meta_ntok(m)) : rec;
}

__device__ __forceinline__ uint32_t block_key(int32_t now, int32_t la, uint32_t m, uint32_t off,
                                              const ScoreTab &t, uint32_t &st)
{
    const int kind = t.kind[meta_queue(m)];
    if (kind == SAE_KIND_LOGNORMAL) return key_lognormal(now, la, m, t, st);
    if (kind == SAE_KIND_STRUCTURAL) return key_structural(now, la, m, off, t, st);
    return key_cheap(kind, now, la, m, t, st);
}

// ----------------------------------------------------------------------------
// Launchers (defined in the .hip files).
struct SelectArgs {
    int32_t now, k;
    const int32_t *k_per_inst;
    uint32_t flags;
    int32_t *victims;
    float *scores;
    int32_t *count;
    int32_t *decision;
    int32_t *decision_count;
};

// Arguments of one prefix-match call (sae_prefix_match).
struct PmArgs {
    int n_req, max_len;
    const uint64_t *hashes;
    const int32_t *lens, *inst;
    int32_t now;
    uint32_t flags;
    int32_t *match_len, *matched_ids;
};

hipError_t launch_block_type(const uint8_t *counts, int64_t n, uint8_t *tau, hipStream_t s);
hipError_t launch_recipe_eval(int fn, int64_t n, const float *x, float *y, hipStream_t s);
hipError_t launch_classify(int n, const uint8_t *hint, uint16_t *meta, const int32_t *roles, hipStream_t s);
hipError_t launch_index_build(const DevCtx &c, hipStream_t s);
hipError_t launch_insert(const DevCtx &c, int32_t n, const int32_t *inst, const int32_t *ids,
                         const uint64_t *hash, const int32_t *parent, const int32_t *la,
                         const uint16_t *meta, const uint32_t *off, uint8_t *skip, hipStream_t s);
hipError_t launch_ref(const DevCtx &c, int32_t n, const int32_t *inst, const int32_t *ids,
                      int32_t delta, hipStream_t s);
hipError_t launch_prefix_match(const DevCtx &c, int32_t n_req, int32_t max_len, const uint64_t *hashes,
                               const int32_t *lens, const int32_t *inst, int32_t now, uint32_t flags,
                               int32_t *match_len, int32_t *matched_ids, hipStream_t s);
// Algorithm 4's placement and the touches of a prefix match with SAE_PM_INTERVALS.
hipError_t launch_pm_place(const DevCtx &c, int32_t n_req, int32_t max_len, const int32_t *inst, int32_t now,
                           uint32_t flags, const int32_t *matched_ids, hipStream_t s);
hipError_t launch_ghost_rebuild(const DevCtx &c, hipStream_t s);
hipError_t launch_index_rebuild(const DevCtx &c, hipStream_t s);
// The pool-scan engine's launches.  With pm, the prefix match pm runs first,
// in one launch with the selection's sampling and bounds (the selection then
// sees the pool after the prefix match, as if called after it); *prep_calls
// counts the context's launches of that kind (the device counters they
// advance follow it) and is incremented when one is enqueued.
hipError_t launch_select_scan(const DevCtx &c, const SelectArgs &a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1,
                              const PmArgs *pm = nullptr, uint32_t *prep_calls = nullptr);
hipError_t launch_select_batched(const DevCtx &c, const SelectArgs &a, hipStream_t s);
hipError_t launch_cascade(const DevCtx &c, const SelectArgs &a, hipStream_t s, int set);
// Device address of the no-allocation predictor's buffer on the current device.
hipError_t predict_scratch(float **out);
hipError_t launch_predict(int n, int d, const uint16_t *h, const uint16_t *w1, const float *b1, const float *w2,
                          const float *b2, const float *w3, const float *b3, float *work, float *logit,
                          uint8_t *pred, hipStream_t s);
hipError_t launch_commit(const DevCtx &c, const SelectArgs &a, hipStream_t s);
hipError_t launch_feedback(const DevCtx &c, uint32_t flags, int learn, hipStream_t s);
int scan_grid_x(int n_inst, int N);
bool batched_engine_fits(const DevCtx &c);
