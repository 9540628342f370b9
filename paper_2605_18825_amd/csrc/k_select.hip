// Scoring and selection kernels (Eq. 1-3, Algorithm 1) for gfx950.
//
// Two engines give identical results:
//  * pool scan (any pool size): a sampling kernel estimates, per instance and
//    queue, a key bound that admits a few times k blocks; one streaming pass
//    over the 10-byte-per-block features scores every block and appends the
//    evictable blocks under the bound to a candidate list; one workgroup per
//    (instance, queue) then radix-selects and sorts the exact k smallest
//    (key, id) among the candidates.  If the bound admitted too few (or too
//    many) blocks, that workgroup falls back to an exact radix select that
//    streams the instance's pool again (slow, rare).  A merge kernel forms the
//    Algorithm 1 decision.
//  * batched (pools of <= 65,536 blocks): one workgroup of 1024 threads per
//    instance keeps every key in registers and does scoring, the radix select
//    of all queues, the sort and the merge in one launch.
#include "sae_internal.h"

#define SCAN_THREADS 256
#define SEL_THREADS 1024
#define SAMPLE_WGS 64
#define SAMPLE_CHUNK 1024
#define BATCH_IPT 64  // keys per thread in the batched engine (64 x 1024 = 65,536 blocks)

namespace {

__device__ __forceinline__ int lane_id() { return (int)__lane_id(); }

__device__ __forceinline__ unsigned long long lanemask_lt()
{
    int l = lane_id();
    return (l == 0) ? 0ull : (~0ull >> (64 - l));
}

// Inclusive scan of v over a wave.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v)
{
    int l = lane_id();
#pragma unroll
    for (int d = 1; d < SAE_WAVE; d <<= 1) {
        uint32_t t = __shfl_up(v, d, SAE_WAVE);
        if (l >= d) v += t;
    }
    return v;
}

// ---------------------------------------------------------------------------
// Boundary search over per-queue histograms of one radix digit.
// hist: [nq][SAE_BINS] in LDS.  For every queue with active[q], finds the bin b
// with below(b) < rem[q] <= below(b) + hist[q][b] and returns b, below(b) and
// hist[q][b].  Needs blockDim.x == 1024 (8 queue slots x 128 threads, each
// owning 16 consecutive bins).  seg_tot: LDS scratch of 16 words.
struct Crossing {
    int32_t bin;
    uint32_t below;
    uint32_t cnt;
};

__device__ void find_crossing(const uint32_t *hist, int nq, const uint32_t *rem, const int32_t *active,
                              Crossing *out, uint32_t *seg_tot)
{
    const int tid = threadIdx.x;
    const int q = tid >> 7;
    const int seg = tid & 127;
    uint32_t s = 0;
    if (q < nq) {
        const uint32_t *h = hist + q * SAE_BINS + seg * 16;
#pragma unroll
        for (int i = 0; i < 16; ++i) s += h[i];
    }
    uint32_t incl = wave_incl_scan(s);
    const int w = tid >> 6;
    if (lane_id() == 63) seg_tot[w] = incl;
    __syncthreads();
    if ((w & 1) == 1) incl += seg_tot[w - 1];
    uint32_t excl = incl - s;
    if (q < nq && active[q]) {
        uint32_t r = rem[q];
        if (excl < r && r <= incl) {
            const uint32_t *h = hist + q * SAE_BINS + seg * 16;
            uint32_t run = excl;
            for (int i = 0; i < 16; ++i) {
                uint32_t c = h[i];
                if (run < r && r <= run + c) {
                    out[q].bin = seg * 16 + i;
                    out[q].below = run;
                    out[q].cnt = c;
                    break;
                }
                run += c;
            }
        }
    }
    __syncthreads();
}

// Per-queue radix-select state (LDS).
struct SelState {
    unsigned long long prefix[SAE_MAX_QUEUES];
    uint32_t rem[SAE_MAX_QUEUES];
    int32_t active[SAE_MAX_QUEUES];  // still refining
    int32_t mode[SAE_MAX_QUEUES];    // 0: select none, 1: all, 2: (e >> shift) <= bound
    int32_t shift[SAE_MAX_QUEUES];
    unsigned long long bound[SAE_MAX_QUEUES];
    Crossing cr[SAE_MAX_QUEUES];
    uint32_t seg_tot[16];
    int32_t any_active;
};

__device__ __forceinline__ bool sel_take(const SelState &st, int q, unsigned long long e)
{
    int m = st.mode[q];
    if (m == 1) return true;
    if (m == 2) return (e >> st.shift[q]) <= st.bound[q];
    return false;
}

// Initialise per-queue state from need[q] and the number of evictable blocks.
__device__ void sel_init(SelState &st, int nq, const uint32_t *need, const uint32_t *nev)
{
    int tid = threadIdx.x;
    if (tid < SAE_MAX_QUEUES) {
        st.prefix[tid] = 0;
        st.rem[tid] = 0;
        st.active[tid] = 0;
        st.mode[tid] = 0;
        st.shift[tid] = 0;
        st.bound[tid] = 0;
        if (tid < nq) {
            uint32_t n = need[tid];
            if (n == 0) {
                st.mode[tid] = 0;
            } else if (n >= nev[tid]) {
                st.mode[tid] = 1;
            } else {
                st.active[tid] = 1;
                st.rem[tid] = n;
            }
        }
    }
    __syncthreads();
    if (tid == 0) {
        int a = 0;
        for (int q = 0; q < nq; ++q) a |= st.active[q];
        st.any_active = a;
    }
    __syncthreads();
}

// One refinement step after the histogram of digit (shift, width) was built.
__device__ void sel_step(SelState &st, int nq, int shift, int width, bool last)
{
    int tid = threadIdx.x;
    if (tid < nq && st.active[tid]) {
        Crossing c = st.cr[tid];
        unsigned long long pb = (st.prefix[tid] << width) | (unsigned long long)c.bin;
        if (c.cnt == st.rem[tid] || last) {
            st.mode[tid] = 2;
            st.shift[tid] = shift;
            st.bound[tid] = pb;
            st.active[tid] = 0;
        } else {
            st.prefix[tid] = pb;
            st.rem[tid] -= c.below;
        }
    }
    __syncthreads();
    if (tid == 0) {
        int a = 0;
        for (int q = 0; q < nq; ++q) a |= st.active[q];
        st.any_active = a;
    }
    __syncthreads();
}

// Bitonic sort, ascending, of nseg independent segments of length P (a power
// of two) stored back to back in LDS.
__device__ void bitonic_sort_segments(unsigned long long *a, int nseg, int P)
{
    const int half = P >> 1;
    const int pairs = nseg * half;
    for (int k = 2; k <= P; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int t = threadIdx.x; t < pairs; t += blockDim.x) {
                int sgi = t / half;
                int u = t - sgi * half;
                int lo = ((u / j) * (j << 1)) + (u % j);
                int hi = lo + j;
                unsigned long long *s = a + (long long)sgi * P;
                unsigned long long x = s[lo], y = s[hi];
                bool up = ((lo & k) == 0);
                if ((x > y) == up) {
                    s[lo] = y;
                    s[hi] = x;
                }
            }
            __syncthreads();
        }
    }
}

__device__ __forceinline__ int lower_bound_u64(const unsigned long long *a, int n, unsigned long long e)
{
    int lo = 0, hi = n;
    while (lo < hi) {
        int mid = (lo + hi) >> 1;
        if (a[mid] < e) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

// Algorithm 1 applied k times to one snapshot: the evict-first list first,
// then the other (sorted) lists merged by (key, id).  lists: Q segments of
// `stride` elements (key << 32 | id), cnt[q] valid in each.  Each element's
// rank in the merged order is its own position plus, for every other list,
// the number of smaller elements (binary search); ids are unique, so ranks are
// distinct.  Returns the decision size.
__device__ int merge_decision(const unsigned long long *lists, int stride, const int32_t *cnt, int Q,
                              int qe, int k, int32_t *dec)
{
    int n1 = (qe >= 0) ? min(k, (int)cnt[qe]) : 0;
    for (int j = threadIdx.x; j < n1; j += blockDim.x)
        dec[j] = (int32_t)(uint32_t)(lists[(long long)qe * stride + j] & 0xFFFFFFFFull);
    int rest = k - n1;
    int total = 0;
    for (int q = 0; q < Q; ++q)
        if (q != qe) total += cnt[q];
    if (rest > 0) {
        for (int q = 0; q < Q; ++q) {
            if (q == qe) continue;
            const unsigned long long *Lq = lists + (long long)q * stride;
            for (int j = threadIdx.x; j < cnt[q]; j += blockDim.x) {
                unsigned long long e = Lq[j];
                int rank = j;
                for (int q2 = 0; q2 < Q && rank < rest; ++q2) {
                    if (q2 == q || q2 == qe) continue;
                    rank += lower_bound_u64(lists + (long long)q2 * stride, cnt[q2], e);
                }
                if (rank < rest) dec[n1 + rank] = (int32_t)(uint32_t)(e & 0xFFFFFFFFull);
            }
        }
    }
    return n1 + min(rest, total);
}

__device__ __forceinline__ void commit_bookkeeping(InstState &s, int d, bool commit)
{
    if (!commit) return;
    long long before = s.ev_count;
    long long after = before + d;
    s.ev_before = before;
    s.ev_count = after;
    s.last_d = d;
    if (s.K > 0 && (after / s.K) > (before / s.K)) s.pending = 1;
}

__device__ __forceinline__ int inst_k(const SelectArgs &a, int inst, int max_k)
{
    // device-supplied k is clamped to 0..max_k (every output has max_k slots)
    int k = a.k_per_inst ? a.k_per_inst[inst] : a.k;
    return k < 0 ? 0 : (k > max_k ? max_k : k);
}

// ---------------------------------------------------------------------------
// Pool-scan engine, step 1: sampled histogram of keys -> per-queue key bound.
__global__ void __launch_bounds__(SCAN_THREADS) k_sample(DevCtx c, SelectArgs a)
{
    extern __shared__ uint32_t sh_hist[];  // [Q][SAE_BINS]
    __shared__ ScoreTab tab;
    __shared__ uint32_t last;
    __shared__ uint32_t seg_tot[SCAN_THREADS / SAE_WAVE];
    __shared__ uint32_t found_bin;
    const int inst = blockIdx.y;
    const int Q = c.Q;
    const long long N = c.N;
    const long long base = (long long)inst * N;
    load_score_tab(tab, c.state[inst], c);
    for (int i = threadIdx.x; i < Q * SAE_BINS; i += blockDim.x) sh_hist[i] = 0;
    __syncthreads();

    long long start = ((long long)blockIdx.x * N) / SAMPLE_WGS;
    long long end = (N <= (long long)SAMPLE_WGS * SAMPLE_CHUNK) ? (((long long)blockIdx.x + 1) * N) / SAMPLE_WGS
                                                              : start + SAMPLE_CHUNK;
    uint32_t st = 0;
    for (long long b = start + threadIdx.x; b < end; b += blockDim.x) {
        uint32_t m = c.meta[base + b];
        if (!meta_evictable(m) || meta_queue(m) >= Q) continue;
        uint32_t key = block_key(a.now, c.la[base + b], m, c.off[base + b], tab, st);
        atomicAdd(&sh_hist[meta_queue(m) * SAE_BINS + (key >> (32 - SAE_DIGIT_BITS))], 1u);
    }
    __syncthreads();
    uint32_t *gh = c.shist + (long long)inst * Q * SAE_BINS;
    for (int i = threadIdx.x; i < Q * SAE_BINS; i += blockDim.x) {
        uint32_t v = sh_hist[i];
        if (v) atomicAdd(&gh[i], v);
    }
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) last = (atomicAdd(&c.done[inst], 1u) == SAMPLE_WGS - 1) ? 1u : 0u;
    __syncthreads();
    if (!last) return;
    __threadfence();

    // Last workgroup of this instance: turn the sampled histogram into bounds.
    const long long S = (N <= (long long)SAMPLE_WGS * SAMPLE_CHUNK) ? N : (long long)SAMPLE_WGS * SAMPLE_CHUNK;
    const int kk = inst_k(a, inst, c.max_k);
    for (int q = 0; q < Q; ++q) {
        const volatile uint32_t *hq = gh + q * SAE_BINS;
        // total sampled evictable of queue q
        uint32_t s = 0;
        for (int i = threadIdx.x; i < SAE_BINS; i += blockDim.x) s += hq[i];
        // reduce
        uint32_t incl = wave_incl_scan(s);
        if (lane_id() == 63) seg_tot[threadIdx.x >> 6] = incl;
        __syncthreads();
        uint32_t tot = 0;
        for (int w = 0; w < SCAN_THREADS / SAE_WAVE; ++w) tot += seg_tot[w];
        __syncthreads();
        double f = (double)S / (double)N;
        double est = (double)tot / f;
        double need = fmin((double)kk, est);
        uint32_t bound = 0xFFFFFFFFu;
        if (need > 0.0 && est > 0.5 * (double)c.cand_cap) {
            double nf = need * f;
            uint32_t r = (uint32_t)ceil(nf * 1.5 + 4.0 * sqrt(nf) + 8.0);
            if (r < tot) {
                // bin where the cumulative sampled count reaches r; 8 bins per thread
                if (threadIdx.x == 0) found_bin = SAE_BINS;
                uint32_t ls = 0;
                int b0 = threadIdx.x * (SAE_BINS / SCAN_THREADS);
                for (int i = 0; i < SAE_BINS / SCAN_THREADS; ++i) ls += hq[b0 + i];
                uint32_t li = wave_incl_scan(ls);
                if (lane_id() == 63) seg_tot[threadIdx.x >> 6] = li;
                __syncthreads();
                uint32_t off = 0;
                for (int w = 0; w < (threadIdx.x >> 6); ++w) off += seg_tot[w];
                uint32_t ex = off + li - ls;
                if (ex < r && r <= ex + ls) {
                    uint32_t run = ex;
                    for (int i = 0; i < SAE_BINS / SCAN_THREADS; ++i) {
                        run += hq[b0 + i];
                        if (run >= r) {
                            found_bin = b0 + i;
                            break;
                        }
                    }
                }
                __syncthreads();
                uint32_t fb = found_bin;
                if (fb < SAE_BINS - 1) bound = ((fb + 1u) << (32 - SAE_DIGIT_BITS)) - 1u;
                __syncthreads();
            }
        }
        if (threadIdx.x == 0) c.thr[(long long)inst * Q + q] = bound;
        __syncthreads();
    }
    for (int i = threadIdx.x; i < Q * SAE_BINS; i += blockDim.x) gh[i] = 0;
    if (threadIdx.x == 0) {
        c.done[inst] = 0;
        set_status(c.status, st);
    }
}

// Pool-scan engine, step 2: one streaming pass over the whole pool.
// Each thread scores 4 consecutive blocks per iteration (16-byte, 8-byte and
// 16-byte loads of last_access, meta and off), counts evictable blocks per
// queue and appends blocks with key <= bound to the candidate lists with one
// atomic per (wave, queue).
__global__ void __launch_bounds__(SCAN_THREADS) k_scan(DevCtx c, SelectArgs a)
{
    __shared__ ScoreTab tab;
    __shared__ uint32_t thr_s[SAE_MAX_QUEUES];
    __shared__ uint32_t nev_s[SAE_MAX_QUEUES];
    __shared__ uint32_t st_s;
    const int inst = blockIdx.y;
    const int Q = c.Q;
    const long long N = c.N;
    const long long base = (long long)inst * N;
    load_score_tab(tab, c.state[inst], c);
    if (threadIdx.x < SAE_MAX_QUEUES) {
        thr_s[threadIdx.x] = (threadIdx.x < Q) ? c.thr[(long long)inst * Q + threadIdx.x] : 0u;
        nev_s[threadIdx.x] = 0;
    }
    if (threadIdx.x == 0) st_s = 0;
    __syncthreads();

    const int now = a.now;
    unsigned long long cnt_lo = 0, cnt_hi = 0;  // 16-bit evictable counters, queues 0-3 / 4-7
    uint32_t st = 0;
    const long long n4 = N >> 2;
    const long long stride = (long long)gridDim.x * blockDim.x;
    const bool vec = ((N & 3) == 0);
    const long long nvec = vec ? n4 : 0;
    unsigned long long *cand_i = c.cand + (long long)inst * Q * c.cand_cap;
    uint32_t *ncand_i = c.n_cand + (long long)inst * Q;

    auto handle = [&](long long b, int32_t la, uint32_t m, uint32_t of) {
        int q = meta_queue(m);
        bool ev = meta_evictable(m) && q < Q;
        uint32_t key = 0;
        if (ev) {
            key = block_key(now, la, m, of, tab, st);
            unsigned long long inc = 1ull << (16 * (q & 3));
            if (q < 4) cnt_lo += inc;
            else cnt_hi += inc;
        }
        bool emit = ev && (key <= thr_s[q]);
        unsigned long long em = __ballot(emit);
        while (em) {
            int l0 = __ffsll((long long)em) - 1;
            int qq = __shfl(q, l0, SAE_WAVE);
            unsigned long long mq = __ballot(emit && q == qq);
            uint32_t basepos = 0;
            if (lane_id() == l0) basepos = atomicAdd(&ncand_i[qq], (uint32_t)__popcll(mq));
            basepos = __shfl(basepos, l0, SAE_WAVE);
            if (emit && q == qq) {
                uint32_t pos = basepos + (uint32_t)__popcll(mq & lanemask_lt());
                if (pos < (uint32_t)c.cand_cap)
                    cand_i[(long long)qq * c.cand_cap + pos] = ((unsigned long long)key << 32) | (uint32_t)b;
            }
            em &= ~mq;
        }
    };

    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i - threadIdx.x < nvec; i += stride) {
        // every lane of a wave runs the same number of iterations (ballots inside)
        bool in = i < nvec;
        int4 la4 = make_int4(0, 0, 0, 0);
        uint2 m4 = make_uint2(0, 0);
        uint4 of4 = make_uint4(0, 0, 0, 0);
        if (in) {
            la4 = reinterpret_cast<const int4 *>(c.la + base)[i];
            m4 = reinterpret_cast<const uint2 *>(c.meta + base)[i];
            of4 = reinterpret_cast<const uint4 *>(c.off + base)[i];
        }
        long long b = i << 2;
        handle(b + 0, la4.x, m4.x & 0xFFFFu, of4.x);
        handle(b + 1, la4.y, m4.x >> 16, of4.y);
        handle(b + 2, la4.z, m4.y & 0xFFFFu, of4.z);
        handle(b + 3, la4.w, m4.y >> 16, of4.w);
    }
    // scalar path (pools whose size is not a multiple of 4)
    if (!vec) {
        for (long long b = (long long)blockIdx.x * blockDim.x + threadIdx.x; b - threadIdx.x < N; b += stride) {
            bool in = b < N;
            uint32_t m = in ? (uint32_t)c.meta[base + b] : 0u;
            int32_t la = in ? c.la[base + b] : 0;
            uint32_t of = in ? c.off[base + b] : 0u;
            handle(b, la, m, of);
        }
    }
    for (int q = 0; q < Q; ++q) {
        uint32_t v = (uint32_t)(((q < 4 ? cnt_lo : cnt_hi) >> (16 * (q & 3))) & 0xFFFFull);
        if (v) atomicAdd(&nev_s[q], v);
    }
    if (st) atomicOr(&st_s, st);
    __syncthreads();
    if (threadIdx.x < Q && nev_s[threadIdx.x]) atomicAdd(&c.n_ev[(long long)inst * Q + threadIdx.x], nev_s[threadIdx.x]);
    if (threadIdx.x == 0) set_status(c.status, st_s);
}

// Pool-scan engine, step 3: exact k smallest (key, id) of one (instance,
// queue) from its candidates (or, if the bound failed, from the whole pool).
__global__ void __launch_bounds__(SEL_THREADS) k_select(DevCtx c, SelectArgs a, int P)
{
    extern __shared__ unsigned long long sh_list[];  // [P] then hist [SAE_BINS] u32
    uint32_t *hist = reinterpret_cast<uint32_t *>(sh_list + P);
    __shared__ SelState st;
    __shared__ ScoreTab tab;
    __shared__ uint32_t need_s, nev_s, lcount, use_fb;
    const int inst = blockIdx.y;
    const int q = blockIdx.x;
    const int Q = c.Q;
    const long long iq = (long long)inst * Q + q;
    const long long N = c.N;
    const long long base = (long long)inst * N;
    if (threadIdx.x == 0) {
        uint32_t nev = c.n_ev[iq];
        uint32_t nc = c.n_cand[iq];
        int kk = inst_k(a, inst, c.max_k);
        uint32_t need = (uint32_t)min((long long)kk, (long long)nev);
        need_s = need;
        nev_s = nev;
        lcount = 0;
        bool fb = (a.flags & SAE_SS_FORCE_FALLBACK) || nc < need || nc > (uint32_t)c.cand_cap;
        use_fb = fb ? 1u : 0u;
        if (fb && need > 0) set_status(c.status, SAE_ST_SELECT_FALLBACK);
    }
    load_score_tab(tab, c.state[inst], c);
    __syncthreads();
    const uint32_t need = need_s;
    const bool fb = use_fb != 0;
    const uint32_t nc = fb ? 0u : c.n_cand[iq];
    const unsigned long long *cand = c.cand + iq * c.cand_cap;
    uint32_t dummy = 0;

    // element source: candidates, or every evictable block of queue q
    auto for_each = [&](auto &&fn) {
        if (!fb) {
            for (uint32_t i = threadIdx.x; i < nc; i += blockDim.x) fn(cand[i]);
        } else {
            for (long long b = threadIdx.x; b < N; b += blockDim.x) {
                uint32_t m = c.meta[base + b];
                if (!meta_evictable(m) || meta_queue(m) != q) continue;
                uint32_t key = block_key(a.now, c.la[base + b], m, c.off[base + b], tab, dummy);
                fn(((unsigned long long)key << 32) | (uint32_t)b);
            }
        }
    };

    // The candidate set holds every evictable block with key <= bound, so the
    // need smallest of the queue are the need smallest candidates.  Count of
    // the element universe for sel_init: candidates (or all evictable).
    uint32_t univ = fb ? nev_s : nc;
    uint32_t needv[SAE_MAX_QUEUES], nevv[SAE_MAX_QUEUES];
    needv[0] = need;
    nevv[0] = univ;
    sel_init(st, 1, needv, nevv);
    // composite (key << 32 | id): digits of 11, 11, 11, 11, 11 and 9 bits
    for (int p = 0; p < 6 && st.any_active; ++p) {
        const int s = (p < 5) ? 53 - 11 * p : 0;
        const int w = (p < 5) ? 11 : 9;
        for (int i = threadIdx.x; i < SAE_BINS; i += blockDim.x) hist[i] = 0;
        __syncthreads();
        const unsigned long long pre = st.prefix[0];
        for_each([&](unsigned long long e) {
            if (p == 0 || (e >> (s + w)) == pre) atomicAdd(&hist[(uint32_t)(e >> s) & ((1u << w) - 1u)], 1u);
        });
        __syncthreads();
        find_crossing(hist, 1, st.rem, st.active, st.cr, st.seg_tot);
        sel_step(st, 1, s, w, p == 5);
    }
    // collect the selection, sort it, write it out
    for (int i = threadIdx.x; i < P; i += blockDim.x) sh_list[i] = ~0ull;
    __syncthreads();
    for_each([&](unsigned long long e) {
        if (sel_take(st, 0, e)) {
            uint32_t pos = atomicAdd(&lcount, 1u);
            if (pos < (uint32_t)P) sh_list[pos] = e;
        }
    });
    __syncthreads();
    bitonic_sort_segments(sh_list, 1, P);
    const int out = (int)min(need, (uint32_t)P);
    const long long ob = iq * c.max_k;
    for (int j = threadIdx.x; j < out; j += blockDim.x) {
        unsigned long long e = sh_list[j];
        a.victims[ob + j] = (int32_t)(uint32_t)(e & 0xFFFFFFFFull);
        if (a.scores) a.scores[ob + j] = __uint_as_float((uint32_t)(e >> 32));
        c.sel[ob + j] = e;
    }
    if (threadIdx.x == 0) {
        a.count[iq] = out;
        c.sel_count[iq] = out;
        c.n_ev[iq] = 0;
        c.n_cand[iq] = 0;
        set_status(c.status, dummy);
    }
}

// Pool-scan engine, step 4: Algorithm 1 decision of each instance.
__global__ void __launch_bounds__(SEL_THREADS) k_merge(DevCtx c, SelectArgs a)
{
    __shared__ int32_t cnt[SAE_MAX_QUEUES];
    const int inst = blockIdx.x;
    const int Q = c.Q;
    if (threadIdx.x < Q) cnt[threadIdx.x] = c.sel_count[(long long)inst * Q + threadIdx.x];
    __syncthreads();
    int kk = inst_k(a, inst, c.max_k);
    int d = merge_decision(c.sel + (long long)inst * Q * c.max_k, c.max_k, cnt, Q, c.ef_queue, kk,
                           a.decision + (long long)inst * c.max_k);
    if (threadIdx.x == 0) {
        a.decision_count[inst] = d;
        commit_bookkeeping(c.state[inst], d, (a.flags & SAE_SS_COMMIT) != 0);
    }
}

// ---------------------------------------------------------------------------
// Batched engine: one workgroup per instance, keys held in registers.
__global__ void __launch_bounds__(SEL_THREADS) k_batched(DevCtx c, SelectArgs a, int P)
{
    extern __shared__ unsigned long long sh_dyn[];  // hist [Q][SAE_BINS] u32, later lists [Q][P] u64
    uint32_t *hist = reinterpret_cast<uint32_t *>(sh_dyn);
    unsigned long long *lists = sh_dyn;
    __shared__ SelState st;
    __shared__ ScoreTab tab;
    __shared__ uint32_t nev_s[SAE_MAX_QUEUES], need_s[SAE_MAX_QUEUES], lcnt[SAE_MAX_QUEUES];
    __shared__ int32_t cnt_s[SAE_MAX_QUEUES];
    __shared__ uint32_t st_s;
    const int inst = blockIdx.x;
    const int Q = c.Q;
    const int N = c.N;
    const long long base = (long long)inst * N;
    const int tid = threadIdx.x;
    load_score_tab(tab, c.state[inst], c);
    if (tid < SAE_MAX_QUEUES) {
        nev_s[tid] = 0;
        lcnt[tid] = 0;
    }
    if (tid == 0) st_s = 0;
    __syncthreads();

    uint32_t key[BATCH_IPT];
    uint32_t info[BATCH_IPT / 8];  // 4 bits per block: 0 = not evictable, else queue + 1
    uint32_t stbits = 0;
#pragma unroll
    for (int g = 0; g < BATCH_IPT / 8; ++g) info[g] = 0;
#pragma unroll
    for (int j = 0; j < BATCH_IPT; ++j) {
        int b = tid + j * SEL_THREADS;
        key[j] = 0;
        // keep the compiler from hoisting every group's loads (register pressure)
        if ((j & 7) == 0) __builtin_amdgcn_sched_barrier(0);
        if (b < N) {
            uint32_t m = c.meta[base + b];
            if (meta_evictable(m) && meta_queue(m) < Q) {
                key[j] = block_key(a.now, c.la[base + b], m, c.off[base + b], tab, stbits);
                int q = meta_queue(m);
                info[j >> 3] |= (uint32_t)(q + 1) << (4 * (j & 7));
                atomicAdd(&nev_s[q], 1u);
            }
        }
    }
    if (stbits) atomicOr(&st_s, stbits);
    __syncthreads();
    if (tid < Q) {
        int kk = inst_k(a, inst, c.max_k);
        need_s[tid] = (uint32_t)min((long long)kk, (long long)nev_s[tid]);
    }
    __syncthreads();
    sel_init(st, Q, need_s, nev_s);

    // composite (key << 16 | id): 48 bits, digits of 11, 11, 11, 11 and 4 bits
    for (int p = 0; p < 5 && st.any_active; ++p) {
        const int s = (p < 4) ? 37 - 11 * p : 0;
        const int w = (p < 4) ? 11 : 4;
        for (int i = tid; i < Q * SAE_BINS; i += blockDim.x) hist[i] = 0;
        __syncthreads();
#pragma unroll
        for (int j = 0; j < BATCH_IPT; ++j) {
            int qi = (int)((info[j >> 3] >> (4 * (j & 7))) & 15u);
            if (qi) {
                int q = qi - 1;
                unsigned long long e = ((unsigned long long)key[j] << 16) | (uint32_t)(tid + j * SEL_THREADS);
                if (st.active[q] && (p == 0 || (e >> (s + w)) == st.prefix[q]))
                    atomicAdd(&hist[q * SAE_BINS + ((uint32_t)(e >> s) & ((1u << w) - 1u))], 1u);
            }
        }
        __syncthreads();
        find_crossing(hist, Q, st.rem, st.active, st.cr, st.seg_tot);
        sel_step(st, Q, s, w, p == 4);
    }
    // collect (the histogram area is reused for the lists)
    for (int i = tid; i < Q * P; i += blockDim.x) lists[i] = ~0ull;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < BATCH_IPT; ++j) {
        int qi = (int)((info[j >> 3] >> (4 * (j & 7))) & 15u);
        if (qi) {
            int q = qi - 1;
            uint32_t id = (uint32_t)(tid + j * SEL_THREADS);
            unsigned long long e = ((unsigned long long)key[j] << 16) | id;
            if (sel_take(st, q, e)) {
                uint32_t pos = atomicAdd(&lcnt[q], 1u);
                if (pos < (uint32_t)P) lists[q * P + pos] = ((unsigned long long)key[j] << 32) | id;
            }
        }
    }
    __syncthreads();
    bitonic_sort_segments(lists, Q, P);
    if (tid < Q) cnt_s[tid] = (int32_t)min(need_s[tid], (uint32_t)P);
    __syncthreads();
    for (int q = 0; q < Q; ++q) {
        const long long ob = ((long long)inst * Q + q) * c.max_k;
        for (int j = tid; j < cnt_s[q]; j += blockDim.x) {
            unsigned long long e = lists[q * P + j];
            a.victims[ob + j] = (int32_t)(uint32_t)(e & 0xFFFFFFFFull);
            if (a.scores) a.scores[ob + j] = __uint_as_float((uint32_t)(e >> 32));
            c.sel[ob + j] = e;
        }
    }
    if (tid < Q) {
        a.count[(long long)inst * Q + tid] = cnt_s[tid];
        c.sel_count[(long long)inst * Q + tid] = cnt_s[tid];
    }
    int kk = inst_k(a, inst, c.max_k);
    int d = merge_decision(lists, P, cnt_s, Q, c.ef_queue, kk, a.decision + (long long)inst * c.max_k);
    if (tid == 0) {
        a.decision_count[inst] = d;
        commit_bookkeeping(c.state[inst], d, (a.flags & SAE_SS_COMMIT) != 0);
        set_status(c.status, st_s);
    }
}

// Kernels whose dynamic LDS may exceed 64 KiB ask for it explicitly.
hipError_t allow_lds(const void *fn, size_t bytes)
{
    if (bytes <= 64 * 1024) return hipSuccess;
    return hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

int pow2_at_least(int x)
{
    int p = 1;
    while (p < x) p <<= 1;
    return p;
}

}  // namespace

bool batched_engine_fits(const DevCtx &c)
{
    if (c.N > BATCH_IPT * SEL_THREADS) return false;
    long long P = pow2_at_least(c.max_k);
    long long lds = (long long)c.Q * (P * 8 > SAE_BINS * 4 ? P * 8 : SAE_BINS * 4);
    return lds <= 128 * 1024;
}

hipError_t launch_select_scan(const DevCtx &c, const SelectArgs &a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1)
{
    // step 1: sampled bounds
    size_t lds_sample = (size_t)c.Q * SAE_BINS * sizeof(uint32_t);
    hipLaunchKernelGGL(k_sample, dim3(SAMPLE_WGS, c.n_inst), dim3(SCAN_THREADS), lds_sample, s, c, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // step 2: streaming pass; 8 workgroups of 256 threads per CU over 256 CUs
    long long n4 = ((long long)c.N + 3) / 4;
    long long want = (n4 + SCAN_THREADS - 1) / SCAN_THREADS;
    int grid_x = (int)(want < 2048 ? want : 2048);
    if (c.n_inst > 1) grid_x = (int)(want < (2048 / c.n_inst + 1) ? want : (2048 / c.n_inst + 1));
    if (grid_x < 1) grid_x = 1;
    if (ev0 && (e = hipEventRecord(ev0, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_scan, dim3(grid_x, c.n_inst), dim3(SCAN_THREADS), 0, s, c, a);
    e = hipGetLastError();
    if (e == hipSuccess && ev1) e = hipEventRecord(ev1, s);
    if (e != hipSuccess) return e;
    // step 3: per (queue, instance) exact select
    int P = pow2_at_least(c.max_k);
    size_t lds_sel = (size_t)P * sizeof(unsigned long long) + SAE_BINS * sizeof(uint32_t);
    if ((e = allow_lds((const void *)k_select, lds_sel)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_select, dim3(c.Q, c.n_inst), dim3(SEL_THREADS), lds_sel, s, c, a, P);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return hipSuccess;
}

hipError_t launch_merge(const DevCtx &c, const SelectArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_merge, dim3(c.n_inst), dim3(SEL_THREADS), 0, s, c, a);
    return hipGetLastError();
}

hipError_t launch_select_batched(const DevCtx &c, const SelectArgs &a, hipStream_t s)
{
    int P = pow2_at_least(c.max_k);
    size_t per = (size_t)P * 8 > (size_t)SAE_BINS * 4 ? (size_t)P * 8 : (size_t)SAE_BINS * 4;
    size_t lds = (size_t)c.Q * per;
    hipError_t e = allow_lds((const void *)k_batched, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_batched, dim3(c.n_inst), dim3(SEL_THREADS), lds, s, c, a, P);
    return hipGetLastError();
}
