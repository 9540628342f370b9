// Strict prefix matching (Sec. 2.1) over the block index: the lookup and the
// workgroup body shared by the prefix-match kernel and the launch that runs a
// prefix match together with the selection's sampling and bounds.
#pragma once

#include "sae_internal.h"

namespace {

// Lookup by linear probing from the home slot.  The probe order is the plain
// one (home, home + 1, ...), but slots are fetched a whole aligned group of
// IDX_GROUP (one 128-byte line) at a time, with every load of the group in
// flight together, so a lookup usually costs one memory round trip.  Tables
// hold at least 64 slots, a multiple of IDX_GROUP.
#define IDX_GROUP 8
__device__ __forceinline__ int index_find(const IndexSlot *tab, uint32_t mask, unsigned long long h, uint32_t *tq)
{
    const uint4 *t4 = reinterpret_cast<const uint4 *>(tab);
    if (SAE_HASH_RESERVED(h)) return -1;
    const int lim = (int)(mask + 1 < (uint32_t)SAE_MAX_PROBES ? mask + 1 : (uint32_t)SAE_MAX_PROBES);
    uint32_t s = hash_home(h, mask);
    int seen = 0;
    while (seen < lim) {
        const uint32_t g = s & ~(uint32_t)(IDX_GROUP - 1);
        uint4 v[IDX_GROUP];
#pragma unroll
        for (int t = 0; t < IDX_GROUP; ++t) v[t] = t4[g + t];
#pragma unroll
        for (int t = 0; t < IDX_GROUP; ++t) {
            if ((uint32_t)t < s - g || seen >= lim) continue;
            ++seen;
            const unsigned long long vh = (unsigned long long)v[t].x | ((unsigned long long)v[t].y << 32);
            if (vh == h) {
                *tq = v[t].w;
                return (int32_t)v[t].z;
            }
            if (vh == SAE_EMPTY_HASH) return -1;
        }
        s = (g + IDX_GROUP) & mask;
    }
    return -1;
}

// Counter field of the prefix match's f-th hit count: queues, then positional
// bins, then block types.
__device__ __forceinline__ int pm_field(int f)
{
    if (f < SAE_MAX_QUEUES) return SAE_CF_HITS + f;
    if (f < SAE_MAX_QUEUES + SAE_N_BINS) return SAE_CF_BHITS + (f - SAE_MAX_QUEUES);
    return SAE_CF_THITS + (f - SAE_MAX_QUEUES - SAE_N_BINS);
}

// ---------------------------------------------------------------------------
// Strict prefix matching (Sec. 2.1), one wave per request.  Lanes probe 64 consecutive
// hashes; the lowest missing lane ends the match and no later chunk is probed.
// queue_hits (and the positional-bin hits of structural blocks) are summed per
// workgroup in LDS (when its requests share an instance) and added into one
// striped counter copy.
// With SAE_PM_INTERVALS the request also finds, per log-normal queue, its
// deepest matched block and stores now - last_access of it (Algorithm 4's
// reuse interval, 0 when none) in pm_rec[r]; no block is touched here, so
// every last_access read is the one from before the call, and k_pm_place
// touches afterwards.
#ifndef PM_FIRST
#define PM_FIRST 8  // hashes of a request's first probe round
#endif
static_assert(PM_FIRST >= 1 && PM_FIRST <= SAE_WAVE, "the first round fits a wave");
#define PM_NC (SAE_MAX_QUEUES + SAE_N_BINS + SAE_N_TYPES)  // queue, bin and type hits
template <int NT>
struct PmShared {
    int32_t winst[NT / SAE_WAVE];
    uint32_t wg_hits[PM_NC];
    uint32_t next;  // requests of the workgroup handed out so far (per_wg > NT / 64)
};

// Hit counts of one wave added into instance inst's counter copy `slot`.
__device__ __forceinline__ void pm_flush(const DevCtx &c, int inst, int slot, const uint32_t (&qcount)[PM_NC])
{
    int32_t *cs = counter_slot(c, inst, slot);
#pragma unroll
    for (int f = 0; f < PM_NC; ++f)
        if (qcount[f] && (f >= SAE_MAX_QUEUES || f < c.Q)) atomicAdd(cs + pm_field(f), (int)qcount[f]);
}

// Workgroup wg of a prefix-match launch of NT-thread workgroups: requests
// wg * per_wg .. (wg + 1) * per_wg - 1.  Wave w takes request w of them; with
// MANY (per_wg > NT / 64), the waves that finish first take the rest, one at
// a time, from a counter in LDS, so that a workgroup lasts about as long as
// its longest request rather than the sum of unlucky pairs.  A wave sums its
// hits per instance and adds them to the counters when its instance changes
// or at the end (the workgroup's waves through LDS when they share one
// instance).  All threads call.
template <int NT, bool MANY = false>
__device__ void prefix_match_wg(const DevCtx &c, int wg, const PmArgs &pa, PmShared<NT> &sh,
                                int per_wg = NT / SAE_WAVE)
{
    constexpr int NC = PM_NC;
    const int n_req = pa.n_req, max_len = pa.max_len;
    const uint64_t *hashes = pa.hashes;
    const int32_t *lens = pa.lens, *inst_a = pa.inst;
    const int32_t now = pa.now;
    const uint32_t flags = pa.flags;
    int32_t *match_len = pa.match_len, *matched_ids = pa.matched_ids;
    int32_t *winst = sh.winst;
    uint32_t *wg_hits = sh.wg_hits;
    const int lane = (int)__lane_id();
    const int wave = threadIdx.x / SAE_WAVE;
    const bool intervals = (flags & SAE_PM_INTERVALS) != 0;
    const bool touch = (flags & SAE_PM_TOUCH) && !intervals;
    if (threadIdx.x < NC) wg_hits[threadIdx.x] = 0;
    if (MANY) {
        if (threadIdx.x == 0) sh.next = NT / SAE_WAVE;
        __syncthreads();
    }
    const long long r0 = (long long)wg * per_wg;
    const int r_end = (int)(r0 + per_wg < n_req ? r0 + per_wg : n_req);
    uint32_t qcount[NC];  // hits of this wave's requests of instance winst_w
#pragma unroll
    for (int q = 0; q < NC; ++q) qcount[q] = 0;
    int32_t winst_w = -1;
    int r = (int)(r0 + wave < r_end ? r0 + wave : r_end);
    while (r < r_end) {  // uniform
        const int inst = inst_a ? inst_a[r] : 0;
        const bool inst_ok = inst >= 0 && inst < c.n_inst;
        if (MANY && inst_ok && winst_w >= 0 && inst != winst_w) {
            if ((flags & SAE_PM_STATS) && lane == 0) pm_flush(c, winst_w, wg, qcount);
#pragma unroll
            for (int q = 0; q < NC; ++q) qcount[q] = 0;
        }
        if (inst_ok) winst_w = inst;
        // positional-bin hits are gathered only while the decay-power learner is on
        const uint32_t ilearn = inst_ok ? c.state[inst].learn : 0u;
        const bool bins = (flags & SAE_PM_STATS) && c.struct_mask && (ilearn & SAE_LEARN_DECAY_POWER);
        // hits per block type are gathered only for the text-form token rule
        const bool types = (flags & SAE_PM_STATS) && (ilearn & SAE_LEARN_TOKEN_EMA);
        int32_t deep[SAE_MAX_QUEUES];  // deepest matched block per log-normal queue (-1: none)
#pragma unroll
        for (int q = 0; q < SAE_MAX_QUEUES; ++q) deep[q] = -1;
        int32_t *mid = matched_ids ? matched_ids + (long long)r * max_len : nullptr;
        // the first two rounds' hashes are loaded with the length (indices
        // clamped into the row, so in bounds whatever the length): one round
        // trip before the first probe instead of two
        const uint64_t *hr = hashes + (long long)r * max_len;
        const unsigned long long h0 = hr[lane < max_len ? lane : max_len - 1];
        const unsigned long long h1 = hr[PM_FIRST + lane < max_len ? PM_FIRST + lane : max_len - 1];
        int len = lens[r];
        if (len > max_len) len = max_len;
        if (len < 0) len = 0;
        if (!inst_ok) {
            if (mid)
                for (int j = lane; j < max_len; j += SAE_WAVE) mid[j] = -1;
            if (lane == 0) {
                match_len[r] = 0;
                set_status(c.status, SAE_ST_BAD_BLOCK);
            }
        } else {
            const IndexSlot *tab = c.index + (long long)inst * ((long long)c.index_mask + 1);
            const long long base = (long long)inst * c.N;
            int m = 0;
            int j0 = 0;
            // Rounds of hashes: the first PM_FIRST, then 64 at a time.  The
            // index slot carries the block's queue, type and positional bin,
            // so a round costs one round trip (its probe); the next round's
            // hashes come with this round's probe.  A short first round spares
            // the probes past an early miss (most requests that miss, miss
            // early) for one more round trip on the long matches.
            int w = PM_FIRST;  // lanes of this round
            uint32_t tq = 0;
            int32_t id = (lane < w && lane < len) ? index_find(tab, c.index_mask, h0, &tq) : -1;
            unsigned long long hnext = (w + lane < len) ? h1 : 0ull;
            while (j0 < len) {  // uniform
                const int j = j0 + lane;
                const bool inr = lane < w && j < len;
                const bool miss = inr && (id < 0);
                const unsigned long long mm = __ballot(miss);
                const int first = mm ? (__ffsll((long long)mm) - 1) : w;
                const int lim = min(first, len - j0);
                const bool hit = lane < lim;
                int q = 0, ty = 0;
                uint32_t bin = 0;
                if (hit) {
                    const long long g = base + id;
                    q = (int)((tq >> 3) & 7u);
                    ty = (int)(tq & 7u);
                    if (bins && ((c.struct_mask >> q) & 1u)) bin = tq >> SAE_TQ_BIN_SHIFT;
                    if (touch) {
                        c.la[g] = now;
                        atomicAdd(&c.access_count[g], 1);
                    }
                    if (mid) mid[j] = id;
                } else if (mid && lane < w && j < max_len) {
                    mid[j] = -1;
                }
                if (flags & SAE_PM_STATS) {
#pragma unroll
                    for (int qq = 0; qq < SAE_MAX_QUEUES; ++qq)
                        qcount[qq] += (uint32_t)__popcll(__ballot(hit && q == qq));
                    if (bins) {
                        const bool sh = hit && ((c.struct_mask >> q) & 1u);
#pragma unroll
                        for (int bb = 0; bb < SAE_N_BINS; ++bb)
                            qcount[SAE_MAX_QUEUES + bb] += (uint32_t)__popcll(__ballot(sh && bin == (uint32_t)bb));
                    }
                    if (types) {
#pragma unroll
                        for (int tt = 0; tt < SAE_N_TYPES; ++tt)
                            qcount[SAE_MAX_QUEUES + SAE_N_BINS + tt] +=
                                (uint32_t)__popcll(__ballot(hit && ty == tt));
                    }
                }
                if (intervals) {
#pragma unroll
                    for (int qq = 0; qq < SAE_MAX_QUEUES; ++qq) {
                        if (!((c.ln_mask >> qq) & 1u)) continue;
                        const unsigned long long bm = __ballot(hit && q == qq);
                        if (bm) deep[qq] = __shfl(id, 63 - __clzll((long long)bm));
                    }
                }
                m = j0 + lim;
                j0 += w;
                if (mm || j0 >= len) break;  // uniform
                // this round matched whole: probe the next 64
                w = SAE_WAVE;
                const int jn = j0 + lane;
                id = (jn < len) ? index_find(tab, c.index_mask, hnext, &tq) : -1;
                hnext = (jn + SAE_WAVE < len) ? hr[jn + SAE_WAVE] : 0ull;
            }
            if (mid)
                for (int j = j0 + lane; j < max_len; j += SAE_WAVE) mid[j] = -1;
            if (lane == 0) match_len[r] = m;
            if (intervals && lane < SAE_MAX_QUEUES) {
                int32_t b = -1;
#pragma unroll
                for (int qq = 0; qq < SAE_MAX_QUEUES; ++qq)
                    if (lane == qq) b = deep[qq];
                int32_t rec = 0;
                if (b >= 0) {
                    const long long dt = (long long)now - (long long)c.la[base + b];
                    if (dt >= 1 && dt <= 0x7FFFFFFFll) rec = (int32_t)dt;
                }
                c.pm_rec[(long long)r * SAE_MAX_QUEUES + lane] = rec;
            }
        }
        if (intervals && !inst_ok && lane < SAE_MAX_QUEUES) c.pm_rec[(long long)r * SAE_MAX_QUEUES + lane] = 0;
        if (!MANY) break;
        uint32_t j = 0;
        if (lane == 0) j = atomicAdd(&sh.next, 1u);
        j = __shfl(j, 0, SAE_WAVE);
        r = (int)(r0 + j < r_end ? r0 + j : r_end);
    }
    if (lane == 0) winst[wave] = winst_w;
    __syncthreads();
    if (!(flags & SAE_PM_STATS)) return;
    // one instance for the whole workgroup?  then sum in LDS
    int i0 = -1;
    bool uniform = true;
    for (int w = 0; w < NT / SAE_WAVE; ++w) {
        const int v = winst[w];
        if (v < 0) continue;
        if (i0 < 0) i0 = v;
        else if (v != i0) uniform = false;
    }
    if (i0 < 0) return;
    if (uniform) {
        if (lane == 0 && winst_w >= 0)
#pragma unroll
            for (int qq = 0; qq < NC; ++qq)
                if (qcount[qq]) atomicAdd(&wg_hits[qq], qcount[qq]);
        __syncthreads();
        const int f = threadIdx.x;
        if (f < NC && wg_hits[f] && (f >= SAE_MAX_QUEUES || f < c.Q))
            atomicAdd(counter_slot(c, i0, wg) + pm_field(f), (int)wg_hits[f]);
    } else if (lane == 0 && winst_w >= 0) {
        pm_flush(c, winst_w, wg, qcount);
    }
}

}  // namespace
