// Scoring and selection kernels (Eq. 1-3, Algorithm 1) for gfx950.
//
// Two engines give identical results:
//  * pool scan (any pool size): a sampling kernel scores a sample of every
//    instance; per (instance, queue) a key bound that admits about 1.25 k
//    blocks and ~k/64-block buckets below it are read off the sorted sample;
//    one streaming pass over the 10-byte-per-block features scores every block
//    and drops the evictable blocks under the bound into their buckets; one
//    workgroup per bucket sorts it and writes the part of it that falls among
//    the k smallest (key, id).  If the bound admitted too few blocks (or a
//    bucket cannot be sorted), the merge kernel recomputes that queue's list
//    by an exact radix select that streams the pool again (slow, rare), then
//    forms the Algorithm 1 decision.
//  * batched (pools of <= 65,536 blocks): one workgroup of 1024 threads per
//    instance keeps every key in registers and does scoring, the radix select
//    of all queues, the sort and the merge in one launch.
#include <hip/hip_ext.h>

#include "sae_internal.h"
#include "pm_match.h"

#define SCAN_THREADS 256
#define SEL_THREADS 1024
#define SAMPLE_WGS SAE_SAMPLE_WGS
#define SAMPLE_CHUNK SAE_SAMPLE_CHUNK
#define BATCH_IPT 64  // blocks per thread of the batched engine (64 x 1024 = 65,536 blocks per instance)

namespace {

__device__ __forceinline__ int lane_id() { return (int)__lane_id(); }

// Workgroup barrier that orders LDS accesses only: global loads and stores
// still in flight stay in flight (__syncthreads waits for them too).
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

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
    lds_barrier();
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
    lds_barrier();
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
    lds_barrier();
    if (tid == 0) {
        int a = 0;
        for (int q = 0; q < nq; ++q) a |= st.active[q];
        st.any_active = a;
    }
    lds_barrier();
}

// One refinement step after the histogram of digit (shift, width) was built.
// The selection is complete when the elements below the crossing bin and the
// bin itself are exactly the ones still needed: then every element whose
// digits up to this one are at most the bin's is taken.
__device__ void sel_step(SelState &st, int nq, int shift, int width, bool last)
{
    int tid = threadIdx.x;
    if (tid < nq && st.active[tid]) {
        Crossing c = st.cr[tid];
        unsigned long long pb = (st.prefix[tid] << width) | (unsigned long long)c.bin;
        if (c.below + c.cnt == st.rem[tid] || last) {
            st.mode[tid] = 2;
            st.shift[tid] = shift;
            st.bound[tid] = pb;
            st.active[tid] = 0;
        } else {
            st.prefix[tid] = pb;
            st.rem[tid] -= c.below;
        }
    }
    lds_barrier();
    if (tid == 0) {
        int a = 0;
        for (int q = 0; q < nq; ++q) a |= st.active[q];
        st.any_active = a;
    }
    lds_barrier();
}

// Bitonic sort, ascending, of nseg independent segments of length P (a power
// of two) that start `stride` elements apart in LDS.  Index arithmetic by
// shifts and masks.
__device__ void bitonic_sort_segments(unsigned long long *a, int nseg, int P, int stride)
{
    if (P < 2) return;
    const int lp = 31 - __clz(P);
    const int lh = lp - 1;
    const int pairs = nseg << lh;
    for (int lk = 1; lk <= lp; ++lk) {
        for (int lj = lk - 1; lj >= 0; --lj) {
            for (int t = threadIdx.x; t < pairs; t += blockDim.x) {
                const int sgi = t >> lh;
                const int u = t & ((1 << lh) - 1);
                const int lo = ((u >> lj) << (lj + 1)) | (u & ((1 << lj) - 1));
                const int hi = lo + (1 << lj);
                unsigned long long *sg = a + (long long)sgi * stride;
                const unsigned long long x = sg[lo], y = sg[hi];
                const bool up = ((lo >> lk) & 1) == 0;
                if ((x > y) == up) {
                    sg[lo] = y;
                    sg[hi] = x;
                }
            }
            lds_barrier();
        }
    }
}

// Sort of P (a power of two, 256 <= P, 2P <= capacity) 64-bit keys in LDS,
// ascending, by a 1024-thread workgroup: each wave sorts runs of 256 keys held
// 4 per lane with a bitonic network (register swaps for strides 1-2, lane
// shuffles above: no barrier), then runs are merged pairwise by merge path
// (each thread finds its split by binary search and merges P/1024 outputs),
// ping-ponging between a[0..P) and a[P..2P).  The result ends in a[0..P).
__device__ __forceinline__ unsigned long long shfl_xor_u64(unsigned long long x, int m)
{
    const uint32_t lo = __shfl_xor((uint32_t)x, m, SAE_WAVE);
    const uint32_t hi = __shfl_xor((uint32_t)(x >> 32), m, SAE_WAVE);
    return ((unsigned long long)hi << 32) | lo;
}

__device__ void wave_sort256(unsigned long long *run)
{
    const int lane = lane_id();
    unsigned long long x[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) x[r] = run[lane * 4 + r];
#pragma unroll
    for (int lk = 1; lk <= 8; ++lk) {
#pragma unroll
        for (int lj = lk - 1; lj >= 0; --lj) {
            const int j = 1 << lj;
            if (j >= 4) {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int e = lane * 4 + r;
                    const unsigned long long y = shfl_xor_u64(x[r], j >> 2);
                    const bool asc = ((e >> lk) & 1) == 0;
                    const bool lower = (e & j) == 0;
                    const unsigned long long mn = x[r] < y ? x[r] : y;
                    const unsigned long long mx = x[r] < y ? y : x[r];
                    x[r] = (lower == asc) ? mn : mx;
                }
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int r2 = r ^ j;
                    if (r < r2) {
                        const int e = lane * 4 + r;
                        const bool asc = ((e >> lk) & 1) == 0;
                        if ((x[r] > x[r2]) == asc) {
                            const unsigned long long t = x[r];
                            x[r] = x[r2];
                            x[r2] = t;
                        }
                    }
                }
            }
        }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) run[lane * 4 + r] = x[r];
}

__device__ void sort_lds(unsigned long long *a, int P)
{
    const int tid = threadIdx.x;
    const int wave = tid / SAE_WAVE;
    const int nwaves = blockDim.x / SAE_WAVE;
    for (int rI = wave; rI < P / 256; rI += nwaves) wave_sort256(a + rI * 256);
    lds_barrier();
    unsigned long long *src = a, *dst = a + P;
    const int E = P / (int)blockDim.x > 0 ? P / (int)blockDim.x : 1;
    for (int run = 256; run < P; run <<= 1) {
        const int o0 = tid * E;
        if (o0 < P) {
            const int pair = o0 / (2 * run);
            const int d = o0 - pair * 2 * run;
            const unsigned long long *A = src + pair * 2 * run;
            const unsigned long long *B = A + run;
            int lo = d > run ? d - run : 0, hi = d < run ? d : run;
            while (lo < hi) {  // split: i from A, d - i from B
                const int mid = (lo + hi) >> 1;
                if (A[mid] < B[d - mid - 1]) lo = mid + 1;
                else hi = mid;
            }
            int i = lo, jb = d - lo;
            unsigned long long *D = dst + pair * 2 * run + d;
            for (int e = 0; e < E; ++e) {
                const bool takeA = (jb >= run) || (i < run && A[i] < B[jb]);
                D[e] = takeA ? A[i++] : B[jb++];
            }
        }
        lds_barrier();
        unsigned long long *t = src;
        src = dst;
        dst = t;
    }
    if (src != a) {
        for (int i = tid; i < P; i += blockDim.x) a[i] = src[i];
        lds_barrier();
    }
}

// Sort of T / S independent segments of S (a power of two, 256 <= S) 64-bit
// keys each, stored back to back in LDS at a[0..T), with a[T..2T) as scratch:
// the runs of 256 sorted as in sort_lds, then merged pairwise inside each
// segment (a pair never crosses a segment's end), 4 outputs per thread per
// round.  All threads call.
__device__ void sort_segments_lds(unsigned long long *a, int T, int S)
{
    const int tid = threadIdx.x;
    const int wave = tid / SAE_WAVE;
    const int nwaves = blockDim.x / SAE_WAVE;
    for (int rI = wave; rI < T / 256; rI += nwaves) wave_sort256(a + rI * 256);
    lds_barrier();
    unsigned long long *src = a, *dst = a + T;
    constexpr int E = 4;
    for (int run = 256; run < S; run <<= 1) {
        for (int o0 = tid * E; o0 < T; o0 += (int)blockDim.x * E) {
            const int pair = o0 / (2 * run);
            const int d = o0 - pair * 2 * run;
            const unsigned long long *A = src + pair * 2 * run;
            const unsigned long long *B = A + run;
            int lo = d > run ? d - run : 0, hi = d < run ? d : run;
            while (lo < hi) {  // split: i from A, d - i from B
                const int mid = (lo + hi) >> 1;
                if (A[mid] < B[d - mid - 1]) lo = mid + 1;
                else hi = mid;
            }
            int i = lo, jb = d - lo;
            unsigned long long *D = dst + pair * 2 * run + d;
            for (int e = 0; e < E; ++e) {
                const bool takeA = (jb >= run) || (i < run && A[i] < B[jb]);
                D[e] = takeA ? A[i++] : B[jb++];
            }
        }
        lds_barrier();
        unsigned long long *t = src;
        src = dst;
        dst = t;
    }
    if (src != a) {
        for (int i = tid; i < T; i += blockDim.x) a[i] = src[i];
        lds_barrier();
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

// Algorithm 1 applied k times to one snapshot: the evict-first list first
// (copied unless copy1 is false: the caller wrote it), then the other (sorted)
// lists merged by (key, id).  lists: Q segments of
// `stride` elements (key << 32 | id), cnt[q] valid in each.  Each element's
// rank in the merged order is its own position plus, for every other list,
// the number of smaller elements (binary search); ids are unique, so ranks are
// distinct.  Returns the decision size.
__device__ int merge_decision(const unsigned long long *lists, int stride, const int32_t *cnt, int Q,
                              int qe, int k, int32_t *dec, bool copy1 = true)
{
    int n1 = (qe >= 0) ? min(k, (int)cnt[qe]) : 0;
    for (int j0 = threadIdx.x; copy1 && j0 < n1; j0 += 8 * blockDim.x) {  // loads first, then stores
        unsigned long long v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int j = j0 + u * (int)blockDim.x;
            v[u] = (j < n1) ? lists[(long long)qe * stride + j] : 0ull;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int j = j0 + u * (int)blockDim.x;
            if (j < n1) dec[j] = (int32_t)(uint32_t)(v[u] & 0xFFFFFFFFull);
        }
    }
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

// Ascending sort of n distinct elements src[0..n) (LDS) into dst[0..n) (LDS):
// each element's position is the number of smaller elements, counted with
// reads that every lane of a wave makes at the same address.  All threads call.
__device__ void rank_sort(const unsigned long long *src, int n, unsigned long long *dst)
{
    for (int t = threadIdx.x; t < n; t += blockDim.x) {
        const unsigned long long e = src[t];
        int rank = 0, i = 0;
        for (; i + 8 <= n; i += 8) {
#pragma unroll
            for (int u = 0; u < 8; ++u) rank += (src[i + u] < e) ? 1 : 0;
        }
        for (; i < n; ++i) rank += (src[i] < e) ? 1 : 0;
        dst[rank] = e;
    }
    lds_barrier();
}

// LDS working set of the per-(instance, queue) selection kernels.
#define LCAP 16384  // elements (128 KiB of LDS)

// Scratch for lds_select_bound and lds_select_rank (LDS).
#define SEL_PIVOTS 64
#define SEL_TMP 1024
struct BoundScratch {
    uint32_t hist[SAE_BINS];
    uint32_t wsum[SEL_THREADS / SAE_WAVE];
    unsigned long long mn, mx;
    uint32_t bin, below, cnt;
    unsigned long long piv[SEL_PIVOTS], tmp[SEL_TMP], res;
    uint32_t pcnt[SEL_PIVOTS + 1], kb, kbelow, kn, fill;
    uint32_t nsorted;  // when nonzero, the nsorted smallest elements, ascending, at tmp + SEL_HEAD
};
#define SEL_HEAD 256  // where the sorted head starts in tmp; at most SEL_HEAD elements
static_assert(SEL_TMP >= 2 * SEL_HEAD, "a head and its sorted copy fit the scratch");

// The n <= SEL_HEAD elements src[0 .. n) (LDS), sorted into b.tmp + SEL_HEAD
// (each placed by its count of smaller ones).  All threads call.
__device__ void lds_sort_head(const unsigned long long *src, int n, BoundScratch &b)
{
    if (threadIdx.x == 0) b.nsorted = (uint32_t)n;
    rank_sort(src, n, b.tmp + SEL_HEAD);
}

// Among n distinct elements held in LDS, a bound B such that exactly `need`
// of them are <= B (1 <= need < n).  Radix select with 11-bit digits starting
// below the common prefix of the smallest and largest element (a run of equal
// keys costs only the digits where the ids differ); it stops at the first
// digit whose crossing bin ends exactly at the need-th element, and returns
// that bin's upper edge.  All threads call; blockDim.x a multiple of 64.
__device__ unsigned long long lds_select_bound(const unsigned long long *el, int n, uint32_t need, BoundScratch &b)
{
    const int tid = threadIdx.x;
    const int nt = blockDim.x;
    const int lane = lane_id();
    const int wave = tid / SAE_WAVE;
    if (tid == 0) {
        b.mn = ~0ull;
        b.mx = 0;
    }
    lds_barrier();
    unsigned long long mn = ~0ull, mx = 0;
    for (int i = tid; i < n; i += nt) {
        const unsigned long long e = el[i];
        mn = e < mn ? e : mn;
        mx = e > mx ? e : mx;
    }
    for (int d = 32; d > 0; d >>= 1) {
        const unsigned long long o1 = __shfl_xor(mn, d, SAE_WAVE), o2 = __shfl_xor(mx, d, SAE_WAVE);
        mn = o1 < mn ? o1 : mn;
        mx = o2 > mx ? o2 : mx;
    }
    if (lane == 0) {
        atomicMin(&b.mn, mn);
        atomicMax(&b.mx, mx);
    }
    lds_barrier();
    mn = b.mn;
    mx = b.mx;
    if (mn == mx) return mn;
    int sh = 64 - __clzll((long long)(mn ^ mx));
    unsigned long long prefix = mn >> sh;
    uint32_t rem = need;
    while (true) {
        const int w = sh < SAE_DIGIT_BITS ? sh : SAE_DIGIT_BITS;
        sh -= w;
        const int nb = 1 << w;
        for (int i = tid; i < nb; i += nt) b.hist[i] = 0;
        lds_barrier();
        for (int i = tid; i < n; i += nt) {
            const unsigned long long e = el[i];
            if ((sh + w >= 64) || (e >> (sh + w)) == prefix) atomicAdd(&b.hist[(uint32_t)(e >> sh) & (nb - 1)], 1u);
        }
        lds_barrier();
        // the bin holding the rem-th element: block scan, each thread owning `per` bins
        const int per = (nb + nt - 1) / nt;
        uint32_t s = 0;
        for (int j = 0; j < per; ++j) {
            const int bi = tid * per + j;
            s += (bi < nb) ? b.hist[bi] : 0u;
        }
        const uint32_t inc = wave_incl_scan(s);
        if (lane == 63) b.wsum[wave] = inc;
        lds_barrier();
        uint32_t run = inc - s;
        for (int w2 = 0; w2 < wave; ++w2) run += b.wsum[w2];
        if (run < rem && rem <= run + s) {
            for (int j = 0; j < per; ++j) {
                const int bi = tid * per + j;
                const uint32_t v = (bi < nb) ? b.hist[bi] : 0u;
                if (run < rem && rem <= run + v) {
                    b.bin = (uint32_t)bi;
                    b.below = run;
                    b.cnt = v;
                }
                run += v;
            }
        }
        lds_barrier();
        const uint32_t bin = b.bin, below = b.below, cnt = b.cnt;
        lds_barrier();
        prefix = (prefix << w) | (unsigned long long)bin;
        rem -= below;
        if (cnt == rem || sh == 0) break;
    }
    return (sh == 0) ? prefix : ((prefix << sh) | ((1ull << sh) - 1ull));
}

// The r-th smallest (1 <= r <= n) of n distinct elements held in LDS.
// Sample select: SEL_PIVOTS elements taken at evenly spaced positions are
// ranked into sorted pivots, every element is counted into the pivot interval
// it falls in, and only the interval holding the r-th element is ranked
// exactly.  When that interval and the ones below it hold at most SEL_HEAD
// elements (a small r: the usual case of a candidate bound), all of them are
// sorted instead, and b.nsorted says how many b.tmp + SEL_HEAD then holds in
// order (0 otherwise); so are all n elements when n <= SEL_HEAD.  An interval
// too large for the scratch falls back to the radix select.  All threads
// call; blockDim.x a multiple of 64 and >= 128.
__device__ unsigned long long lds_select_rank(const unsigned long long *el, int n, uint32_t r, BoundScratch &b)
{
    const int tid = threadIdx.x;
    const int nt = blockDim.x;
    const int lane = lane_id();
    if (n <= SEL_HEAD) {
        lds_sort_head(el, n, b);
        return b.tmp[SEL_HEAD + r - 1];
    }
    if (tid < SAE_WAVE) {
        // pivots: one element per lane from evenly spaced positions, ranked within the wave
        const unsigned long long p = el[(int)(((long long)tid * n) / SEL_PIVOTS)];
        b.tmp[tid] = p;
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        __builtin_amdgcn_wave_barrier();
        uint32_t rk = 0;
#pragma unroll
        for (int i = 0; i < SEL_PIVOTS; ++i) rk += (b.tmp[i] < p) ? 1u : 0u;
        b.piv[rk] = p;
    }
    if (tid < SEL_PIVOTS + 1) b.pcnt[tid] = 0;
    if (tid == 0) b.fill = 0;
    lds_barrier();
    // four elements per thread per round, their searches interleaved
    for (int i0 = tid; i0 < n; i0 += 4 * nt) {
        unsigned long long e[4];
        int k[4];  // pivots below e
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int i = i0 + u * nt;
            e[u] = (i < n) ? el[i] : 0ull;
            k[u] = 0;
        }
#pragma unroll
        for (int st = 32; st > 0; st >>= 1) {
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (b.piv[k[u] + st - 1] < e[u]) k[u] += st;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            k[u] += (b.piv[SEL_PIVOTS - 1] < e[u] && k[u] == SEL_PIVOTS - 1) ? 1 : 0;
            if (i0 + u * nt < n) atomicAdd(&b.pcnt[k[u]], 1u);
        }
    }
    lds_barrier();
    if (tid < SAE_WAVE) {
        // the interval holding the r-th element (interval SEL_PIVOTS counted by lane 63)
        const uint32_t v = b.pcnt[tid] + ((tid == SAE_WAVE - 1) ? b.pcnt[SEL_PIVOTS] : 0u);
        const uint32_t inc = wave_incl_scan(v);
        const uint32_t ex = inc - v;
        if (ex < r && r <= inc) {
            // lane 63 owns two intervals: split them
            if (tid == SAE_WAVE - 1 && r > ex + b.pcnt[tid]) {
                b.kb = SEL_PIVOTS;
                b.kbelow = ex + b.pcnt[tid];
                b.kn = b.pcnt[SEL_PIVOTS];
            } else {
                b.kb = (uint32_t)tid;
                b.kbelow = ex;
                b.kn = b.pcnt[tid];
            }
        }
    }
    lds_barrier();
    const uint32_t kb = b.kb, kbelow = b.kbelow, kn = b.kn;
    if (tid == 0) b.nsorted = 0;
    if (kbelow + kn <= SEL_HEAD) {
        // every element up to the interval's upper pivot, sorted
        const unsigned long long phi = (kb == SEL_PIVOTS) ? ~0ull : b.piv[kb];
        for (int i0 = tid; i0 < n; i0 += 4 * nt) {
            unsigned long long e[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) e[u] = (i0 + u * nt < n) ? el[i0 + u * nt] : ~0ull;
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (i0 + u * nt < n && e[u] <= phi) b.tmp[atomicAdd(&b.fill, 1u)] = e[u];
        }
        lds_barrier();
        lds_sort_head(b.tmp, (int)(kbelow + kn), b);
        return b.tmp[SEL_HEAD + r - 1];
    }
    if (kn > SEL_TMP) {
        lds_barrier();
        const unsigned long long B = lds_select_bound(el, n, r, b);  // exactly r elements <= B
        // the r-th smallest is the largest element <= B
        if (tid == 0) b.mx = 0;
        lds_barrier();
        unsigned long long mx = 0;
        for (int i = tid; i < n; i += nt) mx = (el[i] <= B && el[i] > mx) ? el[i] : mx;
        for (int d = 32; d > 0; d >>= 1) {
            const unsigned long long o = __shfl_xor(mx, d, SAE_WAVE);
            mx = o > mx ? o : mx;
        }
        if (lane == 0) atomicMax(&b.mx, mx);
        lds_barrier();
        return b.mx;
    }
    const unsigned long long plo = (kb == 0) ? 0ull : b.piv[kb - 1];
    const unsigned long long phi = (kb == SEL_PIVOTS) ? ~0ull : b.piv[kb];
    for (int i0 = tid; i0 < n; i0 += 4 * nt) {
        unsigned long long e[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) e[u] = (i0 + u * nt < n) ? el[i0 + u * nt] : 0ull;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const bool in = i0 + u * nt < n && (kb == 0 || plo < e[u]) && e[u] <= phi;
            if (in) b.tmp[atomicAdd(&b.fill, 1u)] = e[u];
        }
    }
    lds_barrier();
    const uint32_t want = r - kbelow - 1;
    for (int t = tid; t < (int)kn; t += nt) {
        const unsigned long long e = b.tmp[t];
        uint32_t rk = 0, i = 0;
        for (; i + 8 <= kn; i += 8) {
#pragma unroll
            for (int u = 0; u < 8; ++u) rk += (b.tmp[i + u] < e) ? 1u : 0u;
        }
        for (; i < kn; ++i) rk += (b.tmp[i] < e) ? 1u : 0u;
        if (rk == want) b.res = e;
    }
    lds_barrier();
    return b.res;
}

// ---------------------------------------------------------------------------
// Pool-scan engine, step 1: score a sample of every instance and record, per
// sampling workgroup ("chunk"), the (key << 32 | id) of every evictable
// sampled block grouped by queue, with the count per queue.  A pool of at most
// SAMPLE_WGS * SAMPLE_CHUNK blocks is sampled whole, a larger one as
// SAMPLE_WGS * SAMPLE_CHUNK / 4 groups of four consecutive blocks spread
// evenly over it: a sample without long runs of consecutive ids keeps the
// buckets of an id-ordered queue (equal keys) small.
struct SampleShared {
    ScoreTab tab;
    unsigned long long tmp[SAMPLE_CHUNK];
    uint8_t tq[SAMPLE_CHUNK];
    uint32_t qcnt[SAE_MAX_QUEUES], qoff[SAE_MAX_QUEUES], qfill[SAE_MAX_QUEUES];
    uint32_t pos_s, st_s;
};

// Chunk `chunk` of instance inst, one sampled block per thread t = 0 ..
// SAMPLE_CHUNK - 1 of a part of the workgroup.  Every thread of the workgroup
// calls (the barriers are the workgroup's), each part with its own chunk and
// shared state; a part with active false only takes the barriers.
__device__ void sample_chunk(const DevCtx &c, const SelectArgs &a, int inst, int chunk, int t, SampleShared &sh,
                             bool active = true)
{
    ScoreTab &tab = sh.tab;
    unsigned long long *tmp = sh.tmp;
    uint8_t *tq = sh.tq;
    uint32_t *qcnt = sh.qcnt, *qoff = sh.qoff, *qfill = sh.qfill;
    uint32_t &pos_s = sh.pos_s, &st_s = sh.st_s;
    const int Q = c.Q;
    const long long N = c.N;
    const long long base = (long long)inst * N;
    long long b = -1;
    if (!active) {
        // no block
    } else if (N <= (long long)SAMPLE_WGS * SAMPLE_CHUNK) {
        const long long start = ((long long)chunk * N) / SAMPLE_WGS;
        const long long end = (((long long)chunk + 1) * N) / SAMPLE_WGS;  // end - start <= SAMPLE_CHUNK
        if (start + t < end) b = start + t;
    } else {
        const long long G = (long long)SAMPLE_WGS * SAMPLE_CHUNK / 4;
        const long long g = (long long)chunk * (SAMPLE_CHUNK / 4) + (t >> 2);
        b = (g * N) / G + (t & 3);  // N / G > 4, so b < N
    }
    uint32_t m = 0, off = 0;
    int32_t la = 0;
    if (b >= 0) {
        m = c.meta[base + b];
        la = c.la[base + b];
        off = c.off[base + b];
    }
    load_score_tab(tab, c.state[inst], c, t);
    if (t < SAE_MAX_QUEUES) {
        qcnt[t] = 0;
        qfill[t] = 0;
    }
    if (t == 0) {
        pos_s = 0;
        st_s = 0;
    }
    lds_barrier();
    uint32_t st = 0;
    const int q = meta_queue(m);
    if (b >= 0 && meta_evictable(m) && q < Q) {
        const uint32_t key = block_key(a.now, la, m, off, tab, st);
        atomicAdd(&qcnt[q], 1u);
        const uint32_t p = atomicAdd(&pos_s, 1u);  // p < SAMPLE_CHUNK: one slot per sampled block
        tmp[p] = ((unsigned long long)key << 32) | (uint32_t)b;
        tq[p] = (uint8_t)q;
    }
    if (st) atomicOr(&st_s, st);
    lds_barrier();
    if (t == 0) {
        uint32_t o = 0;
        for (int qq = 0; qq < SAE_MAX_QUEUES; ++qq) {
            qoff[qq] = o;
            o += qcnt[qq];
        }
    }
    if (active && t < SAE_MAX_QUEUES)
        c.samp_qn[((long long)inst * SAMPLE_WGS + chunk) * SAE_MAX_QUEUES + t] = qcnt[t];
    lds_barrier();
    // the chunk's region holds queue 0's elements, then queue 1's, ...
    const long long reg = ((long long)inst * SAMPLE_WGS + chunk) * SAMPLE_CHUNK;
    const uint32_t n = pos_s;
    for (uint32_t p = t; p < n; p += SAMPLE_CHUNK) {
        const int qq = tq[p];
        const uint32_t pos = qoff[qq] + atomicAdd(&qfill[qq], 1u);
        c.samp[reg + pos] = tmp[p];
    }
    if (t == 0) set_status(c.status, st_s);
}

static_assert(SCAN_THREADS == SAMPLE_CHUNK, "one sampled block per thread");
__global__ void __launch_bounds__(SCAN_THREADS) k_sample(DevCtx c, SelectArgs a)
{
    __shared__ SampleShared sh;
    sample_chunk(c, a, blockIdx.y, blockIdx.x, threadIdx.x, sh);
}

__device__ __forceinline__ int pow2_ge(int x)
{
    return x <= 1 ? 1 : 1 << (32 - __clz(x - 1));
}

// Fixed-step binary searches: every step is unrolled, so that the searches of
// the several elements one thread holds overlap instead of running one after
// the other.
// Last index l < n with a[l] <= x, for a non-decreasing a with a[0] <= x, n <= 2^LOG.
template <int LOG>
__device__ __forceinline__ int last_le(const uint32_t *a, int n, uint32_t x)
{
    int l = 0;
#pragma unroll
    for (int st = 1 << (LOG - 1); st > 0; st >>= 1)
        if (l + st < n && a[l + st] <= x) l += st;
    return l;
}

// Sample rank r of the candidate bound: with f the sampled fraction and need
// the expected number of victims, ceil(1.25 f need + 3 sqrt(f need) + 6): the
// pool then holds about 1.25 need plus a few standard deviations of evictable
// blocks at or below the r-th smallest sampled (key, id).
__device__ __forceinline__ uint32_t bound_rank(double need, double f)
{
    const double nf = need * f;
    return (uint32_t)ceil(nf * 1.25 + 3.0 * sqrt(nf) + 6.0);
}

__device__ __forceinline__ double sample_fraction(long long N)
{
    const long long S = (N <= (long long)SAMPLE_WGS * SAMPLE_CHUNK) ? N : (long long)SAMPLE_WGS * SAMPLE_CHUNK;
    return (double)S / (double)N;
}

// Filter entry of the pool scan for one (type, queue) (see k_scan):
//  x  log-normal: blocks with dt < x lie above the bound (lognormal_dt_floor);
//     0 for the other kinds
//  y  structural / recency: bits of awl = fl(fl(alpha_q w_tau) (1 - 2^-6)) of
//     the product test, 0 (no pruning) unless 2^-90 <= awl <= 2^100
//  z  bits of the bound's key T for the product test: +inf (no pruning)
//     unless T = 0 or 2^-100 <= T < +inf, and for a structural queue gamma = 1
//  w  bit 0: not the evict-first queue; bit 1: recency (p = 1)
// Outside those ranges a subnormal or overflowing product could break the
// test's rounding argument, so nothing is pruned there.
__device__ uint4 scan_entry(int kind, uint32_t dlo, float aw, uint32_t tk, float gamma)
{
    uint4 e = make_uint4(0u, 0u, 0u, 1u);
    if (kind == SAE_KIND_LOGNORMAL) {
        e.x = dlo;
    } else if (kind == SAE_KIND_STRUCTURAL || kind == SAE_KIND_RECENCY) {
        const float awl = aw * (1.0f - 0x1p-6f);
        const float T = __uint_as_float(tk);
        const bool aw_ok = awl >= 0x1p-90f && awl <= 0x1p100f;
        const bool t_ok = tk < 0x7F800000u && (tk == 0u || T >= 0x1p-100f) &&
                          (kind == SAE_KIND_RECENCY || gamma == 1.0f);
        e.y = aw_ok ? __float_as_uint(awl) : 0u;
        e.z = t_ok ? tk : 0x7F800000u;
        e.w = (kind == SAE_KIND_RECENCY) ? 3u : 1u;
    } else {
        e.w = 0u;  // evict-first: the id limit decides
    }
    return e;
}

// Scan pruning of a log-normal queue q for blocks of type ty: the smallest
// D in [0, 2^31] such that every block of (q, ty) with dt < D has a key above
// the bound key tk (IEEE bits of T >= 0), so the scan need not score it.
// D is the first dt at which key(dt) <= bits(T') holds, T' = max(T (1 + 2^-15),
// 2^-100), found by a 64-way bisection with the scan's own key function.
// Why this is safe: for a fixed (q, ty), while P (Eq. 3) stays a normal
// number, this fp32 recipe never gives a larger dt a P more than a factor
// 1 + 2^-19 above a smaller dt's -- ln rises monotonically over every float
// >= 1, the erfc realisation rises by at most one ulp (2^-23 relative) over
// any interval of [0, 9] (both checked exhaustively), and every other step
// is a monotone rounding.  The predecessor D - 1 fails the predicate, so
// P(D - 1) > T' >= 2^-100 (normal) and every dt <= D - 1 has
// P > T' / (1 + 2^-19) > T.  Returns 0 (nothing pruned) when T is not finite
// or a parameter is out of range.  Called by a whole wave; the result is
// wave-uniform.
__device__ uint32_t lognormal_dt_floor(const ScoreTab &t, int q, int ty, uint32_t tk)
{
    const float aw = t.aw[q][ty], mu = t.mu[q], cc = t.c[q];
    const float inf = __uint_as_float(0x7F800000u);
    if (tk >= 0x7F800000u || !(aw >= 0.0f && aw < inf) || !(fabsf(mu) < inf) || !(cc > 0.0f && cc < inf)) return 0;
    const float tp = fmaxf(__uint_as_float(tk) * (1.0f + 0x1p-15f), 0x1p-100f);
    const uint32_t tpb = __float_as_uint(tp);
    if (tpb >= 0x7F800000u) return 0;
    const uint32_t m = (uint32_t)q | ((uint32_t)ty << 3);
    const uint32_t lane = (uint32_t)lane_id();
    uint32_t lo = 0, hi = 0x80000000u;  // the predicate fails at lo (dt = 0 gives +inf) and holds at hi
    uint32_t dummy = 0;
    while (hi - lo > 1) {
        const uint32_t p = lo + (uint32_t)(((unsigned long long)(hi - lo) * (lane + 1)) >> 6);  // lane 63: hi
        const bool ok = (p >= hi) || key_lognormal((int32_t)p, 0, m, t, dummy) <= tpb;
        const unsigned long long mk = __ballot(ok);
        const int f = __ffsll((long long)mk) - 1;
        const uint32_t nhi = __shfl(p, f, SAE_WAVE);
        const uint32_t prev = __shfl(p, (f + SAE_WAVE - 1) & (SAE_WAVE - 1), SAE_WAVE);
        lo = (f == 0) ? lo : prev;
        hi = nhi;
    }
    return hi;
}

// Pool-scan engine, step 2: per (instance, queue), the candidate bound and the
// candidate buckets.  The workgroup stages every sampled element of its queue
// in LDS; the bound is their r-th smallest (key, id); a queue that is
// estimated small takes every evictable block, and one the sample missed gets
// a single bucket for all of them.  Bucket upper ends are the sampled elements
// at or below the bound -- all of them up to SAE_NBUCKET - 1, else an evenly
// spread subset -- and the last one is the bound.  Also writes the scan's
// filter entries and empties the queue's candidate stripes.
#define ALL_EST 2048.0
static_assert(SAMPLE_WGS <= SAE_WAVE, "the chunks' counts fit one wave");
static_assert(SAMPLE_WGS * SAMPLE_CHUNK <= LCAP, "a queue's sampled elements fit the LDS staging area");
struct SplitShared {
    BoundScratch bs;
    uint32_t cbase[SAMPLE_WGS], cpre[SAMPLE_WGS + 1], nsp_s;
    int32_t nb_s;
    unsigned long long spl[SAE_NBUCKET], spl_raw[SAE_NBUCKET], bound_s;
    ScoreTab tab;
};

// Queue q of instance inst; el: LCAP elements of LDS.  With ready false (the
// sample could not be waited for) the queue gets no candidates, so that the
// exact path computes its list.  All SEL_THREADS threads call.
__device__ void split_queue(const DevCtx &c, const SelectArgs &a, int q, int inst, unsigned long long *el,
                            SplitShared &sh, bool ready)
{
    BoundScratch &bs = sh.bs;
    uint32_t *cbase = sh.cbase, *cpre = sh.cpre;
    uint32_t &nsp_s = sh.nsp_s;
    int32_t &nb_s = sh.nb_s;
    unsigned long long *spl = sh.spl, *spl_raw = sh.spl_raw;
    unsigned long long &bound_s = sh.bound_s;
    ScoreTab &tab = sh.tab;
    const int Q = c.Q;
    const int tid = threadIdx.x;
    const int wave = tid / SAE_WAVE;
    const long long iq = (long long)inst * Q + q;
    load_score_tab(tab, c.state[inst], c);
    if (tid < SAE_WAVE) {
        // chunk tid: where queue q's elements start in its region, and how many
        const bool in = tid < SAMPLE_WGS;
        uint32_t v[SAE_MAX_QUEUES];
        const uint32_t *qn = c.samp_qn + ((long long)inst * SAMPLE_WGS + (in ? tid : 0)) * SAE_MAX_QUEUES;
#pragma unroll
        for (int qq = 0; qq < SAE_MAX_QUEUES; ++qq) v[qq] = qn[qq];
        uint32_t o = 0, cnt = 0;
#pragma unroll
        for (int qq = 0; qq < SAE_MAX_QUEUES; ++qq) {
            o += (qq < q) ? v[qq] : 0u;
            cnt = (qq == q) ? v[qq] : cnt;
        }
        cnt = in ? cnt : 0u;
        const uint32_t inc = wave_incl_scan(cnt);
        if (in) {
            cbase[tid] = o;
            cpre[tid] = inc - cnt;
        }
        if (tid == SAMPLE_WGS - 1) cpre[SAMPLE_WGS] = inc;
    }
    // this call's candidate stripes start empty
    if (tid <= SAE_STRIPES) c.stripe_n[iq * (SAE_STRIPES + 1) + tid] = 0;
    if (tid == SEL_THREADS - 1) {
        nsp_s = 0;
        nb_s = 0;
        bound_s = 0;
    }
    lds_barrier();
    const uint32_t tot = cpre[SAMPLE_WGS];  // sampled elements of this queue
    const int kq = ready ? inst_k(a, inst, c.max_k) : 0;
    const double f = sample_fraction(c.N);
    const double est = (double)tot / f;
    const uint32_t r = bound_rank(fmin((double)kq, est), f);
    if (kq == 0) {
        // nothing to select: no candidates
    } else if (tot == 0) {
        // the sample holds no block of this queue: all its evictable blocks, one bucket
        if (tid == 0) {
            bound_s = ~0ull;
            spl[0] = ~0ull;
            nb_s = 1;
        }
    } else {
        const bool all = (r >= tot) || (est <= ALL_EST);
        const uint32_t K = tot;  // <= SAMPLE_WGS * SAMPLE_CHUNK <= LCAP
        const unsigned long long *sp = c.samp + (long long)inst * SAMPLE_WGS * SAMPLE_CHUNK;
        // every load in flight together: a thread's elements past K load
        // element K - 1 again (in bounds) and are not stored
        constexpr int SPT = SAMPLE_WGS * SAMPLE_CHUNK / SEL_THREADS;
        const uint32_t rounds = (K + SEL_THREADS - 1) / SEL_THREADS;  // uniform, <= SPT
        unsigned long long ev[SPT];
#pragma unroll
        for (int m = 0; m < SPT; ++m) {
            if ((uint32_t)m < rounds) {
                uint32_t i = (uint32_t)(tid + m * SEL_THREADS);
                i = i < K ? i : K - 1;
                const int ch = last_le<6>(cpre, SAMPLE_WGS, i);  // the chunk holding element i
                ev[m] = sp[(long long)ch * SAMPLE_CHUNK + cbase[ch] + (i - cpre[ch])];
            }
        }
#pragma unroll
        for (int m = 0; m < SPT; ++m) {
            const uint32_t i = (uint32_t)(tid + m * SEL_THREADS);
            if ((uint32_t)m < rounds && i < K) el[i] = ev[m];
        }
        lds_barrier();
        unsigned long long bound;
        uint32_t rr;  // staged elements at or below the bound
        if (all) {
            bound = ~0ull;
            rr = K;
            if (K <= SAE_NBUCKET - 1) lds_sort_head(el, (int)K, bs);
            else if (tid == 0) bs.nsorted = 0;
            lds_barrier();
        } else {  // r < K
            bound = lds_select_rank(el, (int)K, r, bs);
            rr = r;
        }
        // upper ends: the elements <= bound, or every stride-th staged one of them
        const uint32_t stride = rr <= SAE_NBUCKET - 1 ? 1u : (rr + SAE_NBUCKET - 3) / (SAE_NBUCKET - 2);
        const bool sorted = stride == 1u && bs.nsorted >= rr;  // uniform
        int np;
        if (sorted) {
            // the select left the smallest elements in order: the first rr are the ends
            if (tid < (int)rr) spl[tid] = bs.tmp[SEL_HEAD + tid];
            np = (int)rr;
        } else {
            for (uint32_t i = tid; i < K; i += blockDim.x) {
                const unsigned long long e = el[i];
                if (e <= bound && (stride == 1u || (i % stride) == 0u)) {
                    const uint32_t p = atomicAdd(&nsp_s, 1u);
                    if (p < SAE_NBUCKET - 1) spl_raw[p] = e;
                }
            }
            lds_barrier();
            np = nsp_s < SAE_NBUCKET - 1 ? (int)nsp_s : SAE_NBUCKET - 1;
            rank_sort(spl_raw, np, spl);
        }
        lds_barrier();
        if (tid == 0) {
            int nb = np;
            if (nb == 0 || spl[nb - 1] != bound) spl[nb++] = bound;  // the last upper end is the bound
            bound_s = bound;
            nb_s = nb;
        }
        lds_barrier();
        // Few sampled upper ends (small k against the sample): each gap
        // between consecutive ones (the first taken as wide as the second) is
        // cut into F = 4 or 2 equal ranges of (key << 32 | id) values, with
        // F * ends <= 255, so that buckets stay small.  Any ascending ends
        // ending at the bound are valid; these only balance the work.
        const int nb0 = nb_s;
        const int LF = (4 * nb0 <= SAE_NBUCKET - 1) ? 2 : ((2 * nb0 <= SAE_NBUCKET - 1) ? 1 : 0);
        const int F = 1 << LF;
        if (F >= 2) {
            if (tid < nb0) {
                const unsigned long long hi = spl[tid];
                unsigned long long lo;
                if (tid > 0) {
                    lo = spl[tid - 1];
                } else {
                    const unsigned long long w = (nb0 >= 2) ? spl[1] - spl[0] : 0ull;
                    lo = (spl[0] >= w) ? spl[0] - w : 0ull;
                }
                const unsigned long long d = (hi - lo) >> LF;
                for (int j = 1; j < F; ++j) spl_raw[tid * F + j - 1] = lo + d * (unsigned long long)j;
                spl_raw[tid * F + F - 1] = hi;
            }
            lds_barrier();
            if (tid < nb0 * F) spl[tid] = spl_raw[tid];
            if (tid == 0) nb_s = nb0 * F;
        }
    }
    lds_barrier();
    const int nb = nb_s;
    if (tid < nb) c.split[iq * SAE_NBUCKET + tid] = spl[tid];
    if (tid == 0) {
        c.thr[iq] = bound_s;
        c.nsplit[iq] = nb;
    }
    // the scan's filter entries of this queue: one wave per token type
    if (wave < 8) {
        const uint32_t tk = (uint32_t)(bound_s >> 32);
        uint32_t D = 0;
        if (c.kind[q] == SAE_KIND_LOGNORMAL && wave < SAE_N_TYPES) D = lognormal_dt_floor(tab, q, wave, tk);
        if (lane_id() == 0) c.sent[(long long)inst * 64 + wave * 8 + q] = scan_entry(c.kind[q], D, tab.aw[q][wave], tk, tab.gamma);
        // queue indices >= Q select nothing
        if (q == 0 && lane_id() < SAE_MAX_QUEUES && lane_id() >= Q)
            c.sent[(long long)inst * 64 + wave * 8 + lane_id()] = make_uint4(0xFFFFFFFFu, 0u, 0u, 1u);
    }
    // the evict-first queue's id limit per num_tokens value: (num_tokens, id) <= bound
    if ((q == c.ef_queue || (q == 0 && (c.ef_queue < 0 || c.ef_queue >= Q))) && tid < 16) {
        int32_t lim = -1;
        if (q == c.ef_queue) {
            const uint32_t tk = (uint32_t)(bound_s >> 32), ti = (uint32_t)bound_s;
            const uint32_t kb = __float_as_uint((float)(tid + 1));
            lim = (kb < tk) ? 0x7FFFFFFF : ((kb == tk) ? (int32_t)(ti > 0x7FFFFFFFu ? 0x7FFFFFFFu : ti) : -1);
        }
        c.eflim[(long long)inst * 16 + tid] = lim;
    }
}

__global__ void __launch_bounds__(SEL_THREADS) k_split(DevCtx c, SelectArgs a)
{
    extern __shared__ unsigned long long el[];  // [LCAP]
    __shared__ SplitShared sh;
    split_queue(c, a, blockIdx.x, blockIdx.y, el, sh, true);
}

// A prefix match and the next selection's steps 1 and 2 in one launch of
// SEL_THREADS-thread workgroups (one per compute unit, for their LDS), so
// that the sampling and the bounds run while the requests probe the index.
// Workgroups, in this order:
//  * n_inst * PREP_SAMPLE_WGS sampling workgroups, PREP_PARTS chunks each
//    (the rest of their threads idle: fewer chunks per compute unit keep its
//    scattered loads few, and these workgroups end first); each adds 1 to
//    its instance's prep_done counter once its chunks are stored;
//  * the prefix match, per_wg >= SEL_THREADS / 64 requests per workgroup
//    (prefix_match_wg), as many as make the whole grid fit the device at
//    once where that takes at most 64;
//  * n_inst * Q bound workgroups (split_queue), last, as they need the sample:
//    each first waits until its instance's counter reaches `target` (this
//    call's sampling done).
// The wait ends: workgroups start in index order, so every sampling
// workgroup has started before any bound workgroup, and none of them waits
// on anything; a bounded spin still gives up (that queue then takes the
// exact path) rather than wait forever.
// The sample may see last_access from before or after a touch of the
// concurrent prefix match.  That only moves the candidate bound, which
// shapes the work, not the result: the final kernel checks that the
// candidates cover every list and otherwise computes it exactly.
#define PREP_PARTS 2                               // chunks per sampling workgroup
#define PREP_SAMPLE_WGS (SAMPLE_WGS / PREP_PARTS)  // sampling workgroups per instance
#define PREP_SPIN_LIMIT (1u << 18)
static_assert(SAMPLE_WGS % PREP_PARTS == 0 && PREP_PARTS * SAMPLE_CHUNK <= SEL_THREADS, "whole sampling workgroups");
union PrepShared {
    SampleShared s[SEL_THREADS / SAMPLE_CHUNK];
    SplitShared p;
    PmShared<SEL_THREADS> m;
};
__global__ void __launch_bounds__(SEL_THREADS) k_match_prep(DevCtx c, SelectArgs a, PmArgs pa, uint32_t target,
                                                            int n_pm, int per_wg)
{
    extern __shared__ unsigned long long el[];  // [LCAP]
    __shared__ PrepShared sh;
    __shared__ int32_t ready_s;
    const int b = blockIdx.x;
    const int ns = c.n_inst * PREP_SAMPLE_WGS;
    if (b < ns) {
        const int inst = b / PREP_SAMPLE_WGS, part = threadIdx.x / SAMPLE_CHUNK;
        sample_chunk(c, a, inst, (b % PREP_SAMPLE_WGS) * PREP_PARTS + part, threadIdx.x % SAMPLE_CHUNK, sh.s[part],
                     part < PREP_PARTS);
        // every wave's stores reach the L2 before the barrier; thread 0's
        // release then writes the L2 back for the other dies' caches
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (threadIdx.x == 0) {
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
            __hip_atomic_fetch_add(&c.prep_done[inst], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    } else if (b < ns + n_pm) {
        prefix_match_wg<SEL_THREADS, true>(c, b - ns, pa, sh.m, per_wg);
    } else {
        const int inst = (b - ns - n_pm) / c.Q, q = (b - ns - n_pm) % c.Q;
        if (threadIdx.x == 0) {
            int32_t ok = 1;
            uint32_t spins = 0;
            while ((int32_t)(__hip_atomic_load(&c.prep_done[inst], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) -
                             target) < 0) {
                if (++spins > PREP_SPIN_LIMIT) {
                    ok = 0;
                    break;
                }
                __builtin_amdgcn_s_sleep(2);
            }
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            ready_s = ok;
        }
        __syncthreads();
        split_queue(c, a, q, inst, el, sh.p, ready_s != 0);
    }
}

// Pool-scan engine, step 3: one streaming pass over the whole pool.
// Each wave takes batches of SCAN_BATCH consecutive blocks (4 per lane, read
// with 16-, 8- and 16-byte loads of last_access, meta and off), with the
// loads of the next two batches in flight while one is examined.  A cheap
// exact filter drops almost every evictable block whose (key, id) lies above
// its queue's bound without evaluating Eq. 1-3; its table (k_split, one
// 16-byte entry per (type, queue), see scan_entry) makes every test pass
// trivially for the other kinds, so a block costs one table read and no
// branch:
//  * log-normal: dt below the (queue, type) threshold;
//  * structural and recency: the product test (product_prunes);
//  * evict-first: the key is num_tokens, so (key, id) <= bound is an id limit
//    per num_tokens value.
// The blocks that remain (about the bound's candidates) are queued per wave in
// LDS with their features; a wave scores its queue exactly once 64 are queued,
// and at the end the four waves score what is left together.  Blocks with
// (key, id) <= bound are buffered in LDS per queue (one LDS atomic per wave
// and queue); at the end each queue's buffer is appended to one of the
// queue's candidate stripes with a single device atomic, and what does not fit
// that stripe, or the buffer, goes to the queue's overflow list.  Batches of a pool whose
// size is not a multiple of 4, and the last partial batch, take a path with
// per-element loads.
#define SCAN_BATCH 256  // blocks per wave per batch: 4 per lane
#define SCAN_WAVES (SCAN_THREADS / SAE_WAVE)
#define SCAN_LIST (SAE_WAVE + SCAN_BATCH)  // queued blocks per wave
#define SCAN_CB 128  // candidates a workgroup buffers per queue before appending to a stripe

// Structural (pn / pd = 1 - o_b / o_max) and recency (pn = pd = 1) blocks:
// true only if fl(pn awl) > fl(fl(T dt) pd), which implies P > T.  Proof
// sketch, for 2^-90 <= awl <= 2^100 and T = 0 or 2^-100 <= T < +inf (the
// entry disables the test otherwise): the recipe's p = fl(1 - fl(o_b / o_max))
// is at least (pn / pd)(1 - 2^-8)(1 - 2^-24) because pd < 2^16; P =
// fl(fl(aw p) / dt) is at least (pn / pd)(aw / dt)(1 - 2^-8)(1 - 2^-13)
// (1 - 2^-23) even where it is subnormal (it is then above 2^-137); the test's
// own roundings stay in the normal range, so with the factor 1 - 2^-6 in awl
// it implies (pn / pd)(aw / dt) > T (1 + 2^-7), hence P > T.  dt = 0 gives a
// right side of 0 (and P = +inf); T = +inf never prunes.
__device__ __forceinline__ bool product_prunes(uint32_t pn, uint32_t pd, float awl, float tb, int32_t dt)
{
    const float lhs = (float)pn * awl;
    const float rhs = (tb * (float)dt) * (float)pd;
    return lhs > rhs;
}

// Four consecutive blocks of one lane, as loaded from HBM.
struct Quad {
    int4 la;
    uint4 off;
    uint2 m;
};

__device__ __forceinline__ Quad load_quad_vec(const DevCtx &c, long long e0)
{
    Quad r;
    r.la = *reinterpret_cast<const int4 *>(c.la + e0);
    r.m = *reinterpret_cast<const uint2 *>(c.meta + e0);
    r.off = *reinterpret_cast<const uint4 *>(c.off + e0);
    return r;
}

// Elements e0 .. e0 + 3 of the instance starting at `base`, those below N.
__device__ __forceinline__ Quad load_quad_safe(const DevCtx &c, long long base, long long e0, long long N)
{
    uint32_t m[4] = {0, 0, 0, 0};
    int32_t l[4] = {0, 0, 0, 0};
    uint32_t o[4] = {0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if (e0 + j < N) {
            l[j] = c.la[base + e0 + j];
            m[j] = c.meta[base + e0 + j];
            o[j] = c.off[base + e0 + j];
        }
    }
    Quad r;
    r.la = make_int4(l[0], l[1], l[2], l[3]);
    r.off = make_uint4(o[0], o[1], o[2], o[3]);
    r.m = make_uint2(m[0] | (m[1] << 16), m[2] | (m[3] << 16));
    return r;
}

__global__ void __launch_bounds__(SCAN_THREADS) k_scan(DevCtx c, SelectArgs a)
{
    __shared__ ScoreTab tab;
    __shared__ uint4 ent[64];
    __shared__ int32_t ef_lim[16];
    __shared__ unsigned long long thr_s[SAE_MAX_QUEUES];
    __shared__ uint32_t cnt_s[SAE_MAX_QUEUES];
    __shared__ uint32_t st_s;
    __shared__ uint32_t left_s[SCAN_WAVES + 1];
    __shared__ int4 s_lst[SCAN_WAVES][SCAN_LIST];  // queued blocks: last_access, off, meta, id
    __shared__ unsigned long long cbuf[SAE_MAX_QUEUES][SCAN_CB];  // this workgroup's candidates per queue
    __shared__ uint32_t res_base[SAE_MAX_QUEUES], res_n[SAE_MAX_QUEUES], ovf_base[SAE_MAX_QUEUES],
        ovf_n[SAE_MAX_QUEUES];
    const int inst = blockIdx.y;
    const int wg = blockIdx.x;
    const int Q = c.Q;
    const long long N = c.N;
    const long long base = (long long)inst * N;
    const int lane = lane_id();
    const int wave = threadIdx.x / SAE_WAVE;
    const int tid = threadIdx.x;
    const long long nb = (N + SCAN_BATCH - 1) / SCAN_BATCH;
    const long long nfull = ((N & 3) == 0) ? N / SCAN_BATCH : 0;  // batches read with vector loads
    const long long gw = (long long)wg * SCAN_WAVES + wave;
    const long long tw = (long long)gridDim.x * SCAN_WAVES;
    // the first two batches' loads go out before the tables are read
    auto ld = [&](long long bi) {
        const long long b = bi < nfull ? bi : nfull - 1;
        return load_quad_vec(c, base + b * SCAN_BATCH + lane * 4);
    };
    Quad qa = {}, qb = {}, qc = {};
    if (nfull > 0) {
        qa = ld(gw);
        qb = ld(gw + tw);
    }
    load_score_tab(tab, c.state[inst], c);
    if (tid < 64) ent[tid] = c.sent[(long long)inst * 64 + tid];
    if (tid >= 64 && tid < 80) ef_lim[tid - 64] = c.eflim[(long long)inst * 16 + tid - 64];
    if (tid >= 128 && tid < 128 + SAE_MAX_QUEUES) {
        const int q = tid - 128;
        thr_s[q] = (q < Q) ? c.thr[(long long)inst * Q + q] : 0ull;
        cnt_s[q] = 0;
    }
    if (tid == 0) st_s = 0;
    __syncthreads();

    const int now = a.now;
    uint32_t st = 0;
    unsigned long long *cand = c.cand + (long long)inst * Q * 2 * SAE_LCAP;
    uint32_t *stripe_n = c.stripe_n + (long long)inst * Q * (SAE_STRIPES + 1);
    int4 *lst = s_lst[wave];

    // append (key, id) of an evictable block if it is within its queue's bound:
    // to the workgroup's LDS buffer of the queue, or once that is full, straight
    // to the queue's overflow list (one device atomic per wave and queue)
    auto emit = [&](bool act, int q, uint32_t key, uint32_t b) {
        const unsigned long long comp = ((unsigned long long)key << 32) | b;
        const bool e = act && (comp <= thr_s[q]);
        unsigned long long em = __ballot(e);
        while (em) {
            const int l0 = __ffsll((long long)em) - 1;
            const int qq = __shfl(q, l0, SAE_WAVE);
            const unsigned long long mq = __ballot(e && q == qq);
            uint32_t bp = 0;
            if (lane == l0) bp = atomicAdd(&cnt_s[qq], (uint32_t)__popcll(mq));
            bp = __shfl(bp, l0, SAE_WAVE);
            const uint32_t pos = bp + (uint32_t)__popcll(mq & lanemask_lt());
            const bool in_e = e && q == qq;
            if (in_e && pos < SCAN_CB) cbuf[qq][pos] = comp;
            const unsigned long long ms = __ballot(in_e && pos >= SCAN_CB);
            if (ms) {
                const int ls = __ffsll((long long)ms) - 1;
                uint32_t sb = 0;
                if (lane == ls) sb = atomicAdd(&stripe_n[qq * (SAE_STRIPES + 1) + SAE_STRIPES], (uint32_t)__popcll(ms));
                sb = __shfl(sb, ls, SAE_WAVE);
                if (in_e && pos >= SCAN_CB) {
                    const uint32_t sp = sb + (uint32_t)__popcll(ms & lanemask_lt());
                    if (sp < SAE_LCAP) cand[(long long)qq * 2 * SAE_LCAP + SAE_LCAP + sp] = comp;
                }
            }
            em &= ~mq;
        }
    };
    // score one queued block per active lane, then emit it
    auto score = [&](bool act, const int4 v) {
        const uint32_t m = act ? (uint32_t)v.z : 0u;
        const uint32_t key = block_key(now, act ? v.x : now, m, act ? (uint32_t)v.y : 0u, tab, st);
        emit(act, meta_queue(m), key, (uint32_t)v.w);
    };

    const unsigned long long lt = lanemask_lt();
    uint32_t nl = 0;  // queued blocks of this wave (wave-uniform)
    auto process = [&](const Quad &cur, long long bi) {
        const int32_t lav[4] = {cur.la.x, cur.la.y, cur.la.z, cur.la.w};
        const uint32_t offv[4] = {cur.off.x, cur.off.y, cur.off.z, cur.off.w};
        const uint32_t mv[4] = {cur.m.x & 0xFFFFu, cur.m.x >> 16, cur.m.y & 0xFFFFu, cur.m.y >> 16};
        const uint32_t b0 = (uint32_t)(bi * SCAN_BATCH) + (uint32_t)lane * 4u;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t m = mv[j];
            const uint4 e = ent[m & 63u];
            const bool ev = (m & (SAE_META_VALID | SAE_META_LEAF | SAE_META_REF)) == (SAE_META_VALID | SAE_META_LEAF);
            const int32_t dtr = now - lav[j];
            st |= (ev & (dtr < 0)) ? (uint32_t)SAE_ST_FUTURE_ACCESS : 0u;
            const int32_t dt = dtr < 0 ? 0 : dtr;
            const uint32_t ob = offv[j] & 0xFFFFu, om = offv[j] >> 16;
            const bool one = ((e.w & 2u) != 0u) | (om == 0u);
            const uint32_t pn = one ? 1u : (om > ob ? om - ob : 0u);
            const uint32_t pd = one ? 1u : om;
            // every test evaluated (no short-circuit branches)
            const int32_t lim = ef_lim[(m >> SAE_META_NTOK_SHIFT) & 15u];
            const bool k_ef = ((e.w & 1u) != 0u) | ((int32_t)(b0 + j) <= lim);
            const bool k_pr = !product_prunes(pn, pd, __uint_as_float(e.y), __uint_as_float(e.z), dt);
            const bool keep = ev & ((uint32_t)dt >= e.x) & k_pr & k_ef;
            const unsigned long long km = __ballot(keep);
            if (keep) lst[nl + (uint32_t)__popcll(km & lt)] = make_int4(lav[j], (int32_t)offv[j], (int32_t)m, (int32_t)(b0 + j));
            nl += (uint32_t)__popcll(km);
        }
        if (nl >= SAE_WAVE) {  // wave-uniform, rare
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
            __builtin_amdgcn_wave_barrier();
            do {
                nl -= SAE_WAVE;
                score(true, lst[nl + lane]);
            } while (nl >= SAE_WAVE);
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
            __builtin_amdgcn_wave_barrier();
        }
    };

    // full batches: unconditional vector loads, two batches ahead
    for (long long bi = gw; bi < nfull; bi += 3 * tw) {  // wave-uniform
        qc = ld(bi + 2 * tw);
        process(qa, bi);
        if (bi + tw >= nfull) break;
        qa = ld(bi + 3 * tw);
        process(qb, bi + tw);
        if (bi + 2 * tw >= nfull) break;
        qb = ld(bi + 4 * tw);
        process(qc, bi + 2 * tw);
    }
    // the rest: per-element loads
    for (long long bi = nfull + gw; bi < nb; bi += tw)
        process(load_quad_safe(c, base, bi * SCAN_BATCH + lane * 4, N), bi);

    // what the waves left queued, scored by the four waves together
    if (lane == 0) left_s[wave] = nl;
    lds_barrier();
    if (tid == 0) {
        uint32_t o = 0;
        for (int w = 0; w < SCAN_WAVES; ++w) {
            const uint32_t v = left_s[w];
            left_s[w] = o;
            o += v;
        }
        left_s[SCAN_WAVES] = o;
    }
    lds_barrier();
    const uint32_t total = left_s[SCAN_WAVES];
    for (uint32_t i0 = (uint32_t)wave * SAE_WAVE; i0 < total; i0 += SCAN_THREADS) {  // wave-uniform
        const uint32_t i = i0 + (uint32_t)lane;
        int w = 0;
        while (w + 1 < SCAN_WAVES && left_s[w + 1] <= i) ++w;
        const bool act = i < total;
        score(act, act ? s_lst[w][i - left_s[w]] : make_int4(0, 0, 0, 0));
    }
    if (st) atomicOr(&st_s, st);
    lds_barrier();
    // the buffered candidates go to stripe wg mod SAE_STRIPES of their queue
    // (one reservation per queue), the part that does not fit it to the
    // queue's overflow list (a second reservation, rarely); then every thread
    // stores
    const uint32_t stripe = (uint32_t)wg % SAE_STRIPES;
    if (tid < Q) {
        const uint32_t n = min(cnt_s[tid], (uint32_t)SCAN_CB);
        const uint32_t b = n ? atomicAdd(&stripe_n[tid * (SAE_STRIPES + 1) + stripe], n) : 0u;
        const uint32_t fit = b >= SAE_STRIPE_CAP ? 0u : min(n, (uint32_t)SAE_STRIPE_CAP - b);
        res_n[tid] = n;
        res_base[tid] = b;
        ovf_n[tid] = fit;  // buffered candidates that fit the stripe
        ovf_base[tid] = (n > fit) ? atomicAdd(&stripe_n[tid * (SAE_STRIPES + 1) + SAE_STRIPES], n - fit) : 0u;
    }
    if (tid == 0) set_status(c.status, st_s);
    lds_barrier();
    for (int i = tid; i < Q * SCAN_CB; i += SCAN_THREADS) {
        const int q = i / SCAN_CB;
        const uint32_t j = (uint32_t)(i - q * SCAN_CB);
        if (j >= res_n[q]) continue;
        unsigned long long *cq = cand + (long long)q * 2 * SAE_LCAP;
        if (j < ovf_n[q]) {
            cq[stripe * SAE_STRIPE_CAP + res_base[q] + j] = cbuf[q][j];
        } else {
            const uint32_t p = ovf_base[q] + (j - ovf_n[q]);
            if (p < SAE_LCAP) cq[SAE_LCAP + p] = cbuf[q][j];
        }
    }
}

// Pool-scan engine, step 4: the sorted lists and the Algorithm 1 decision, in
// one launch of FIN_THREADS-thread workgroups per instance (the commit, a
// chain of scattered accesses per victim, follows in a kernel that spreads the
// victims over many compute units):
//  * every workgroup first reads each queue's stripe counts, bound and bucket
//    count (one round of loads) and derives the same facts from them: the
//    candidates C_q, the list size need_q = min(k, evictable), whether the
//    queue's candidates are complete (C_q >= need_q, no stripe over its
//    capacity, not forced to the exact path), and the decision's size;
//  * "group" workgroups, FIN_G buckets of one queue each: stream the queue's
//    candidates, count those at or below the group's lower end, rank the
//    ones inside by bucket and write the part within the first need_q
//    positions (the evict-first queue's list also fills the decision's first
//    positions, Algorithm 1 stage 1);
//  * "union" workgroups: the decision's stage 2 is the first k - n1 of all
//    other queues' blocks by (P, id), and every one of them is a candidate of
//    its queue (each lies among its own queue's first k), so ranking the
//    union of those candidates up to the reference bound (the smallest bound
//    among those queues) gives it exactly; the union's ranges are cut at the
//    bucket ends of all those queues merged, so that each holds about the
//    same number of candidates however the queues' keys interleave;
//  * one finisher workgroup writes the list sizes and the decision size and
//    updates the eviction count.  If any queue's candidates are incomplete,
//    every other workgroup stops and the finisher alone computes everything
//    by the exact path (radix select streaming the pool) and merges.
#define FIN_THREADS 1024
#define FIN_G 16                             // buckets per group workgroup
#define FIN_GPQ (SAE_NBUCKET / FIN_G)        // group workgroups per queue
#define FIN_NU 64                            // union workgroups
#define FIN_GCAP 4096                        // candidates a workgroup ranks at once
#define FIN_U (SAE_LCAP / FIN_THREADS)       // candidates per thread of one streamed queue
#define FIN_STACK 80                         // pending ranges (a range splits into two)
#define FIN_SB 64                            // sub-bins per bucket in the ranking
#define FIN_T 64                             // largest segment ranked by comparison alone
#define FIN_RSTACK (FIN_GCAP / FIN_T)        // pending segments (disjoint, each above FIN_T)
#define FIN_MAXREF 48                        // refinements of one range before comparison takes over
static_assert(SAE_STRIPES == SAE_WAVE, "one stripe per lane");
static_assert(FIN_G <= 16, "bucket indices fit the bucket histogram");

struct FinInfo {
    uint32_t C[SAE_MAX_QUEUES];     // candidates held (stripes, then the overflow list)
    uint32_t over[SAE_MAX_QUEUES];  // candidates lost beyond the overflow list's capacity
    uint32_t need[SAE_MAX_QUEUES];  // list size min(k, evictable)
    int32_t nb[SAE_MAX_QUEUES];
    int32_t fail[SAE_MAX_QUEUES];
    unsigned long long thr[SAE_MAX_QUEUES];
    uint32_t spre[SAE_MAX_QUEUES][SAE_STRIPES + 1];  // position of each stripe's first candidate in queue
                                                     // order; [SAE_STRIPES]: the overflow list's
    int32_t any_fail, n1, rest, d;
};

struct FinRange {
    unsigned long long lo, hi;  // range (lo, hi], or [0, hi] when !has_lo
    int32_t has_lo, e0, e1;     // bucket upper ends e0 .. e1 - 1 of the range (e1 - 1 ends at hi), or none
};

// Per-instance facts from the scan's counts (all threads; ends with a barrier).
__device__ void fin_info(const DevCtx &c, const SelectArgs &a, int inst, uint32_t kq, FinInfo &f)
{
    const int Q = c.Q, tid = threadIdx.x, lane = lane_id(), wave = tid / SAE_WAVE;
    if (wave < Q) {
        const long long iq = (long long)inst * Q + wave;
        const uint32_t *sn = c.stripe_n + iq * (SAE_STRIPES + 1);
        const uint32_t raw = sn[lane];
        const uint32_t ovr = sn[SAE_STRIPES];
        const int32_t nb = c.nsplit[iq];
        const unsigned long long thr = c.thr[iq];
        const uint32_t capd = raw < SAE_STRIPE_CAP ? raw : (uint32_t)SAE_STRIPE_CAP;
        const uint32_t inc = wave_incl_scan(capd);
        f.spre[wave][lane] = inc - capd;
        const uint32_t S = __shfl(inc, SAE_WAVE - 1, SAE_WAVE);
        const uint32_t ovk = ovr < SAE_LCAP ? ovr : (uint32_t)SAE_LCAP;
        if (lane == 0) {
            f.spre[wave][SAE_STRIPES] = S;
            f.C[wave] = S + ovk;
            f.over[wave] = ovr - ovk;
            f.nb[wave] = nb;
            f.thr[wave] = thr;
        }
    }
    lds_barrier();
    if (tid == 0) {
        int any = 0;
        uint32_t other = 0, n_ef = 0;
        for (int q = 0; q < Q; ++q) {
            const bool all = f.thr[q] == ~0ull;
            const uint32_t need = (all && f.C[q] < kq) ? f.C[q] : kq;
            const bool fail = need > 0 && ((a.flags & SAE_SS_FORCE_FALLBACK) || f.nb[q] <= 0 || f.C[q] < need ||
                                           f.over[q] > 0 || f.C[q] > SAE_LCAP);
            f.need[q] = need;
            f.fail[q] = fail ? 1 : 0;
            any |= fail ? 1 : 0;
            if (q == c.ef_queue) n_ef = need;
            else other += need;
        }
        f.any_fail = any;
        f.n1 = (int32_t)n_ef;
        f.rest = (int32_t)(kq - n_ef);
        f.d = (int32_t)(n_ef + ((uint32_t)f.rest < other ? (uint32_t)f.rest : other));
    }
    lds_barrier();
}

// Where candidate i (< C) of a queue lies: the stripes in order, then the
// overflow list.  Computed without a branch, so that the loads of all of a
// thread's candidates can be in flight together (a load inside a divergent
// branch is waited for at the branch's end).
__device__ __forceinline__ uint32_t fin_slot(const uint32_t *spre, uint32_t i)
{
    const int s = last_le<6>(spre, SAE_STRIPES, i);
    const uint32_t in_stripe = (uint32_t)s * SAE_STRIPE_CAP + (i - spre[s]);
    const uint32_t ov = spre[SAE_STRIPES];
    return i >= ov ? (uint32_t)SAE_LCAP + (i - ov) : in_stripe;
}

// Ranks the candidates of the queues in `src` (a bit mask) that lie in
// (first range's lo, ends[e1 - 1]]: out(r, e) is called for every one of them
// whose rank r among all those queues' candidates is below `need`.
// Streaming: wave w reads stripes w, w + 16, w + 32, w + 48 of a queue, every
// load issued before any is used, and keeps the candidates inside the range
// in a region of its own (a register count, no atomics).  Ranking, over those
// only: each candidate's bucket, the buckets' smallest and largest values, a
// counting sort by sub-bin (FIN_SB equal value ranges between a bucket's
// smallest and largest value; monotone in the value, so the sub-bins are
// ordered), and inside its sub-bin (a handful of candidates) each one's rank
// by comparison.  Equal keys of many blocks (blocks added together share
// last_access, so a queue's keys repeat in clusters of hundreds) put whole
// clusters into one sub-bin; a sub-bin of more than FIN_T candidates is
// therefore refined by a counting sort of its own over FIN_THREADS sub-bins
// between its smallest and largest value (each refinement puts those two in
// different sub-bins, so segments shrink), until every segment is small.  A
// range holding more than fits is split in two (by its bucket ends, or by
// value once it has a single bucket) and the halves are ranked in order.  All
// threads call; `ends` is in LDS.
template <typename Out>
__device__ void fin_rank(const DevCtx &c, int inst, const FinInfo &f, uint32_t src, const unsigned long long *ends,
                         FinRange first, uint32_t need, unsigned long long *st1, unsigned long long *st2,
                         Out out)
{
    constexpr int NW = FIN_THREADS / SAE_WAVE;
    constexpr int NSB = 16 * FIN_SB;
    constexpr int WCAP = FIN_GCAP / NW;  // staging slots per wave
    constexpr int PER = FIN_GCAP / FIN_THREADS;
    static_assert(NSB == FIN_THREADS, "one sub-bin per thread in the scan");
    static_assert(SAE_STRIPES == 4 * NW && SAE_STRIPE_CAP == 4 * SAE_WAVE, "four stripes of four slots per lane");
    const int tid = threadIdx.x, lane = lane_id(), wave = tid / SAE_WAVE;
    __shared__ FinRange stack[FIN_STACK];
    __shared__ int32_t sp_s, stop_s, go_s, full_s;
    __shared__ uint32_t below_s, wsum[NW], wcnt[NW], wpre[NW + 1];
    __shared__ uint32_t hist[NSB], soff[NSB + 1];
    __shared__ unsigned long long bmin[16], bmax[16];
    __shared__ float sbmul[16];
    __shared__ FinRange cur;
    __shared__ uint32_t segbits[FIN_GCAP / 32];  // bit p: a segment starts at position p
    __shared__ uint2 rstack[FIN_RSTACK];
    __shared__ int32_t rsp_s;
    __shared__ uint32_t rlo_s, rhi_s;
    __shared__ unsigned long long rmin_s, rmax_s;
    if (tid == 0) {
        stack[0] = first;
        sp_s = 1;
        stop_s = 0;
    }
    lds_barrier();
    while (true) {
        if (tid == 0) {
            cur = stack[--sp_s];
            below_s = 0;
            full_s = 0;
        }
        hist[tid] = 0;
        if (tid < 16) {
            bmin[tid] = ~0ull;
            bmax[tid] = 0;
        }
        lds_barrier();
        const FinRange r = cur;
        const bool has_ends = r.e1 > r.e0;
        const int nbk = has_ends ? r.e1 - r.e0 : 1;
        uint32_t below = 0, wn = 0;  // wn: this wave's staged candidates (wave-uniform)
        bool full = false;
        const unsigned long long lt = lanemask_lt();
        unsigned long long *wst = st1 + wave * WCAP;
        auto take = [&](unsigned long long e, bool ok) {
            const bool under = ok && r.has_lo && e <= r.lo;
            below += under ? 1u : 0u;
            const bool inr = ok && !under && e <= r.hi;
            const unsigned long long m = __ballot(inr);
            const uint32_t p = wn + (uint32_t)__popcll(m & lt);
            if (inr && p < WCAP) wst[p] = e;
            wn += (uint32_t)__popcll(m);
        };
        for (int q = 0; q < c.Q; ++q) {
            if (!((src >> q) & 1u)) continue;
            const uint32_t C = f.C[q];
            if (C == 0) continue;  // uniform
            const unsigned long long *cq = c.cand + ((long long)inst * c.Q + q) * 2 * SAE_LCAP;
            const uint32_t *spre = f.spre[q];
            unsigned long long ev[16];
            uint32_t okm = 0;
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                const int st = wave + NW * r4;
                const uint32_t cnt = spre[st + 1] - spre[st];
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const uint32_t j = (uint32_t)(lane + SAE_WAVE * v);
                    ev[r4 * 4 + v] = cq[st * SAE_STRIPE_CAP + (j < cnt ? j : 0u)];
                    okm |= (j < cnt) ? (1u << (r4 * 4 + v)) : 0u;
                }
            }
#pragma unroll
            for (int u = 0; u < 16; ++u) take(ev[u], (okm >> u) & 1u);
            // the overflow list (usually empty), split over the waves
            const uint32_t ov = C - spre[SAE_STRIPES];
            for (uint32_t b0 = 0; b0 < ov; b0 += FIN_THREADS) {
                const uint32_t i = b0 + (uint32_t)tid;
                take(cq[SAE_LCAP + (i < ov ? i : ov - 1)], i < ov);
            }
        }
        full = wn > WCAP;
        for (int o = 32; o > 0; o >>= 1) below += __shfl_xor(below, o, SAE_WAVE);
        if (lane == 0) {
            if (below) atomicAdd(&below_s, below);
            wcnt[wave] = wn < WCAP ? wn : WCAP;
            if (full) full_s = 1;
        }
        lds_barrier();
        if (tid == 0) {
            uint32_t o = 0;
            for (int w = 0; w < NW; ++w) {
                wpre[w] = o;
                o += wcnt[w];
            }
            wpre[NW] = o;
        }
        lds_barrier();
        const uint32_t bl = below_s, n = wpre[NW];
        if (bl >= need) {
            // this range and every later one lie beyond the first `need`
        } else if (full_s) {
            if (tid == 0) {
                FinRange a1 = r, a2 = r;
                if (r.e1 - r.e0 >= 2) {
                    const int mid = (r.e0 + r.e1) / 2;
                    a1.e1 = mid;
                    a1.hi = ends[mid - 1];
                    a2.e0 = mid;
                    a2.lo = ends[mid - 1];
                    a2.has_lo = 1;
                } else {
                    const unsigned long long lo = r.has_lo ? r.lo : 0ull;
                    const unsigned long long m = lo + (r.hi - lo) / 2;
                    a1.e0 = a1.e1 = a2.e0 = a2.e1 = 0;
                    a1.hi = m;
                    a2.lo = m;
                    a2.has_lo = 1;
                }
                if (sp_s + 2 <= FIN_STACK) {
                    stack[sp_s++] = a2;
                    stack[sp_s++] = a1;
                } else {
                    stop_s = 1;  // cannot happen: each split at least halves a 64-bit range
                }
            }
        } else {
            // this thread's staged candidates (position p of the waves' regions in order)
            unsigned long long e4[PER];
            int b4[PER];
#pragma unroll
            for (int u = 0; u < PER; ++u) {
                const uint32_t p = (uint32_t)(tid + u * FIN_THREADS);
                b4[u] = -1;
                if (p < n) {
                    const int w = last_le<4>(wpre, NW, p);
                    e4[u] = st1[w * WCAP + (p - wpre[w])];
                    int b = 0;  // the bucket: ends below e
                    if (has_ends) {
#pragma unroll
                        for (int st = 8; st > 0; st >>= 1)
                            if (b + st < nbk && ends[r.e0 + b + st - 1] < e4[u]) b += st;
                    }
                    b4[u] = b;
                    atomicMin(&bmin[b], e4[u]);
                    atomicMax(&bmax[b], e4[u]);
                }
            }
            lds_barrier();
            if (tid < nbk) sbmul[tid] = (float)FIN_SB / ((float)(bmax[tid] - bmin[tid]) + 1.0f);
            lds_barrier();
            int k4[PER];
#pragma unroll
            for (int u = 0; u < PER; ++u) {
                k4[u] = -1;
                if (b4[u] >= 0) {
                    int sb = (int)((float)(e4[u] - bmin[b4[u]]) * sbmul[b4[u]]);
                    sb = sb < FIN_SB - 1 ? sb : FIN_SB - 1;
                    k4[u] = b4[u] * FIN_SB + sb;
                    atomicAdd(&hist[k4[u]], 1u);
                }
            }
            lds_barrier();
            // counting sort by sub-bin: offsets by a workgroup scan (one sub-bin per thread)
            const uint32_t v = hist[tid];
            const uint32_t inc = wave_incl_scan(v);
            if (lane == SAE_WAVE - 1) wsum[wave] = inc;
            lds_barrier();
            uint32_t pre = 0;
            for (int w = 0; w < wave; ++w) pre += wsum[w];
            soff[tid] = pre + inc - v;
            if (tid == FIN_THREADS - 1) soff[NSB] = pre + inc;
            hist[tid] = 0;  // from here the fill count of the sub-bin
            lds_barrier();
#pragma unroll
            for (int u = 0; u < PER; ++u)
                if (k4[u] >= 0) st2[soff[k4[u]] + atomicAdd(&hist[k4[u]], 1u)] = e4[u];
            if (tid < FIN_GCAP / 32) segbits[tid] = 0;
            if (tid == 0) rsp_s = 0;
            lds_barrier();
            // segments: the non-empty sub-bins; the large ones wait for refinement
            {
                const uint32_t s0 = soff[tid], cnt = soff[tid + 1] - s0;
                if (cnt) atomicOr(&segbits[s0 >> 5], 1u << (s0 & 31));
                if (cnt > FIN_T) rstack[atomicAdd(&rsp_s, 1)] = make_uint2(s0, s0 + cnt);
            }
            lds_barrier();
            // every thread reads the stack size between two barriers, before
            // thread 0 pops, so all of them take the same branch
            bool more = rsp_s > 0;
            for (int nref = 0; more && nref < FIN_MAXREF; ++nref) {  // uniform
                lds_barrier();
                if (tid == 0) {
                    const uint2 sg = rstack[--rsp_s];
                    rlo_s = sg.x;
                    rhi_s = sg.y;
                    rmin_s = ~0ull;
                    rmax_s = 0;
                }
                hist[tid] = 0;
                lds_barrier();
                const uint32_t lo = rlo_s, hi = rhi_s;
                unsigned long long mn = ~0ull, mx = 0;
                for (uint32_t p = lo + tid; p < hi; p += FIN_THREADS) {
                    const unsigned long long e = st2[p];
                    mn = e < mn ? e : mn;
                    mx = e > mx ? e : mx;
                }
                for (int o = 32; o > 0; o >>= 1) {
                    const unsigned long long a2 = shfl_xor_u64(mn, o), b2 = shfl_xor_u64(mx, o);
                    mn = a2 < mn ? a2 : mn;
                    mx = b2 > mx ? b2 : mx;
                }
                if (lane == 0 && lo + (uint32_t)wave * SAE_WAVE < hi) {
                    atomicMin(&rmin_s, mn);
                    atomicMax(&rmax_s, mx);
                }
                lds_barrier();
                const unsigned long long smn = rmin_s;
                const float mul = (float)FIN_THREADS / ((float)(rmax_s - smn) + 1.0f);
                auto sub = [&](unsigned long long e) {
                    const int x = (int)((float)(e - smn) * mul);
                    return x < FIN_THREADS - 1 ? x : FIN_THREADS - 1;
                };
                for (uint32_t p = lo + tid; p < hi; p += FIN_THREADS) atomicAdd(&hist[sub(st2[p])], 1u);
                lds_barrier();
                const uint32_t hv = hist[tid];
                const uint32_t hinc = wave_incl_scan(hv);
                if (lane == SAE_WAVE - 1) wsum[wave] = hinc;
                lds_barrier();
                uint32_t hpre = 0;
                for (int w = 0; w < wave; ++w) hpre += wsum[w];
                soff[tid] = lo + hpre + hinc - hv;
                hist[tid] = 0;
                lds_barrier();
                for (uint32_t p = lo + tid; p < hi; p += FIN_THREADS) {
                    const unsigned long long e = st2[p];
                    const int x = sub(e);
                    st1[soff[x] + atomicAdd(&hist[x], 1u)] = e;
                }
                lds_barrier();
                for (uint32_t p = lo + tid; p < hi; p += FIN_THREADS) st2[p] = st1[p];
                if (hv) {
                    const uint32_t s0 = soff[tid];
                    atomicOr(&segbits[s0 >> 5], 1u << (s0 & 31));
                    if (hv > FIN_T) rstack[atomicAdd(&rsp_s, 1)] = make_uint2(s0, s0 + hv);
                }
                lds_barrier();
                more = rsp_s > 0;
            }
            // rank inside the final segments by comparison
            for (uint32_t p = tid; p < n; p += FIN_THREADS) {
                const unsigned long long e = st2[p];
                uint32_t lo = p, hi = p + 1;
                {  // the segment's first position: the last set bit at or below p
                    int w = (int)(p >> 5);
                    uint32_t bits = segbits[w] & (0xFFFFFFFFu >> (31 - (p & 31)));
                    while (!bits && w > 0) bits = segbits[--w];
                    lo = bits ? (uint32_t)(w * 32 + 31 - __clz(bits)) : 0u;
                }
                if (bl + lo >= need) continue;  // the whole segment lies beyond the first `need`
                {  // its end: the next set bit above p, or n
                    int w = (int)(p >> 5);
                    uint32_t bits = (p & 31) == 31 ? 0u : (segbits[w] & (0xFFFFFFFFu << ((p & 31) + 1)));
                    while (!bits && w + 1 < FIN_GCAP / 32 && (uint32_t)(w + 1) * 32 < n) bits = segbits[++w];
                    hi = bits ? (uint32_t)(w * 32 + __ffs(bits) - 1) : n;
                    hi = hi < n ? hi : n;
                }
                uint32_t rk = 0, i = lo;
                for (; i + 4 <= hi; i += 4) {
#pragma unroll
                    for (int t = 0; t < 4; ++t) rk += (st2[i + t] < e) ? 1u : 0u;
                }
                for (; i < hi; ++i) rk += (st2[i] < e) ? 1u : 0u;
                const uint32_t rank = bl + lo + rk;
                if (rank < need) out(rank, e);
            }
        }
        // thread 0 alone changes the stack, so it decides whether to go on
        if (tid == 0) go_s = !(bl >= need || sp_s == 0 || stop_s);
        lds_barrier();
        if (!go_s) break;  // uniform
    }
}

// The exact path of one instance, run by the finisher alone when some queue's
// candidates are incomplete (or when forced): every queue's list by a radix
// select that streams the pool (its evictable blocks counted first), the
// decision by merging the lists (Algorithm 1).
__device__ void fin_exact(const DevCtx &c, const SelectArgs &a, int inst, uint32_t kq, const FinInfo &f, int P,
                          long long lds_bytes, unsigned long long *el)
{
    __shared__ SelState st;
    __shared__ ScoreTab tab;
    __shared__ int32_t cnt[SAE_MAX_QUEUES];
    __shared__ uint32_t lcount, st_s;
    const int Q = c.Q;
    const int tid = threadIdx.x;
    const int lane = lane_id();
    const long long N = c.N;
    const long long base = (long long)inst * N;
    load_score_tab(tab, c.state[inst], c);
    if (tid == 0) {
        st_s = 0;
        set_status(c.status, SAE_ST_SELECT_FALLBACK);
    }
    __syncthreads();
    uint32_t dummy = 0;
    for (int q = 0; q < Q; ++q) {
        if (tid == 0) lcount = 0;
        __syncthreads();
        {
            uint32_t n = 0;
            for (long long b = tid; b < N; b += blockDim.x) {
                const uint32_t m = c.meta[base + b];
                n += (meta_evictable(m) && meta_queue(m) == q) ? 1u : 0u;
            }
            for (int d = 32; d > 0; d >>= 1) n += __shfl_xor(n, d, SAE_WAVE);
            if (lane == 0 && n) atomicAdd(&lcount, n);
        }
        __syncthreads();
        const uint32_t nev = lcount;
        const uint32_t need = nev < kq ? nev : kq;
        if (tid == 0) {
            const long long iq = (long long)inst * Q + q;
            cnt[q] = (int32_t)need;
            a.count[iq] = (int32_t)need;
            c.sel_count[iq] = (int32_t)need;
            uint32_t *dbg = c.sel_stats + iq * 4;
            dbg[0] = nev;
            dbg[1] = f.C[q];
            dbg[2] = f.over[q];
            dbg[3] = 1;
            lcount = 0;
        }
        __syncthreads();
        if (need == 0) continue;  // uniform
        auto for_each = [&](auto &&fn) {
            for (long long b = tid; b < N; b += blockDim.x) {
                const uint32_t m = c.meta[base + b];
                if (!meta_evictable(m) || meta_queue(m) != q) continue;
                const uint32_t key = block_key(a.now, c.la[base + b], m, c.off[base + b], tab, dummy);
                fn(((unsigned long long)key << 32) | (uint32_t)b);
            }
        };
        uint32_t needv[SAE_MAX_QUEUES], nevv[SAE_MAX_QUEUES];
        needv[0] = need;
        nevv[0] = nev;
        sel_init(st, 1, needv, nevv);
        for (int p = 0; p < 6 && st.any_active; ++p) {
            const int s = (p < 5) ? 53 - 11 * p : 0;
            const int w = (p < 5) ? 11 : 9;
            uint32_t *hist = reinterpret_cast<uint32_t *>(el);
            for (int i = tid; i < SAE_BINS; i += blockDim.x) hist[i] = 0;
            __syncthreads();
            const unsigned long long pre = st.prefix[0];
            for_each([&](unsigned long long e) {
                if (p == 0 || (e >> (s + w)) == pre) atomicAdd(&hist[(uint32_t)(e >> s) & ((1u << w) - 1u)], 1u);
            });
            __syncthreads();
            find_crossing(hist, 1, st.rem, st.active, st.cr, st.seg_tot);
            sel_step(st, 1, s, w, p == 5);
        }
        __syncthreads();
        for_each([&](unsigned long long e) {
            if (sel_take(st, 0, e)) {
                const uint32_t pos = atomicAdd(&lcount, 1u);
                if (pos < (uint32_t)P) el[pos] = e;
            }
        });
        __syncthreads();
        const uint32_t out = need < (uint32_t)P ? need : (uint32_t)P;
        const int PS = P < 256 ? 256 : P;
        for (int i = tid + (int)out; i < PS; i += blockDim.x) el[i] = ~0ull;
        __syncthreads();
        sort_lds(el, PS);
        const long long ob = ((long long)inst * Q + q) * c.max_k;
        for (uint32_t j = tid; j < out; j += blockDim.x) {
            const unsigned long long e = el[j];
            a.victims[ob + j] = (int32_t)(uint32_t)(e & 0xFFFFFFFFull);
            if (a.scores) a.scores[ob + j] = __uint_as_float((uint32_t)(e >> 32));
            c.sel[ob + j] = e;
        }
        __syncthreads();
    }
    if (dummy) atomicOr(&st_s, dummy);
    __syncthreads();
    // stage 2 searches the sorted lists: from LDS when they fit
    const unsigned long long *lists = c.sel + (long long)inst * Q * c.max_k;
    int stride = c.max_k;
    const int n1 = (c.ef_queue >= 0) ? min((int)kq, cnt[c.ef_queue]) : 0;
    int maxc = 0;
    for (int q = 0; q < Q; ++q) maxc = max(maxc, (int)cnt[q]);
    if ((int)kq > n1 && (long long)Q * maxc * 8 <= lds_bytes) {
        for (int i = tid; i < Q * maxc; i += blockDim.x) {
            const int q = i / maxc, j = i - q * maxc;
            if (j < cnt[q]) el[i] = lists[(long long)q * c.max_k + j];
        }
        __syncthreads();
        lists = el;
        stride = maxc;
    }
    int32_t *dec = a.decision + (long long)inst * c.max_k;
    const int d = merge_decision(lists, stride, cnt, Q, c.ef_queue, (int)kq, dec, true);
    if (tid == 0) {
        a.decision_count[inst] = d;
        // a cascading decision is completed (and counted) by k_cascade
        if (!(a.flags & SAE_SS_CASCADE)) commit_bookkeeping(c.state[inst], d, (a.flags & SAE_SS_COMMIT) != 0);
        set_status(c.status, st_s);
    }
}

__global__ void __launch_bounds__(FIN_THREADS) k_final(DevCtx c, SelectArgs a, int P, long long lds_bytes)
{
    extern __shared__ unsigned long long fdyn[];  // staging (group / union) or the exact path's sort
    __shared__ FinInfo f;
    __shared__ unsigned long long ends[FIN_G + 1];
    __shared__ int32_t ref_s;
    const int inst = blockIdx.y;
    const int unit = blockIdx.x;
    const int Q = c.Q;
    const int tid = threadIdx.x;
    const uint32_t kq = (uint32_t)inst_k(a, inst, c.max_k);
    const int n_group = Q * FIN_GPQ;
    if (unit < n_group && tid <= FIN_G) {
        // a group's bucket ends go out with the first round of loads
        const int b0 = (unit % FIN_GPQ) * FIN_G;
        const unsigned long long *spl = c.split + ((long long)inst * Q + unit / FIN_GPQ) * SAE_NBUCKET;
        ends[tid] = (b0 + tid - 1 >= 0) ? spl[b0 + tid - 1] : 0ull;
    }
    // a union workgroup's: every queue's bucket ends (2 per thread, Q <= 8)
    static_assert(SAE_MAX_QUEUES * SAE_NBUCKET == 2 * FIN_THREADS, "two bucket ends per thread");
    unsigned long long uend[2] = {0ull, 0ull};
    if (unit >= n_group && unit < n_group + FIN_NU) {
        const unsigned long long *spl = c.split + (long long)inst * Q * SAE_NBUCKET;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int i = tid + h * FIN_THREADS;
            uend[h] = (i < Q * SAE_NBUCKET) ? spl[i] : 0ull;
        }
    }
    fin_info(c, a, inst, kq, f);
    unsigned long long *st1 = fdyn, *st2 = fdyn + FIN_GCAP;
    int32_t *dec = a.decision + (long long)inst * c.max_k;
    if (unit < n_group + FIN_NU) {
        if (f.any_fail) return;  // uniform: the finisher computes everything
        const bool group = unit < n_group;
        const int q = group ? unit / FIN_GPQ : 0;
        if (!group && tid == 0) {
            // the reference queue: smallest bound among the other queues with a list
            int ref = -1;
            for (int qq = 0; qq < Q; ++qq)
                if (qq != c.ef_queue && f.need[qq] > 0 && (ref < 0 || f.thr[qq] < f.thr[ref])) ref = qq;
            ref_s = ref;
        }
        lds_barrier();
        const int rq = group ? q : ref_s;
        const uint32_t need = group ? f.need[q] : (uint32_t)f.rest;
        if (rq < 0 || need == 0) return;  // uniform
        uint32_t src = 0;
        if (group) {
            src = 1u << q;
        } else {
            for (int qq = 0; qq < Q; ++qq)
                if (qq != c.ef_queue && f.need[qq] > 0) src |= 1u << qq;
        }
        FinRange first;
        if (group) {
            const int nb = f.nb[q];
            const int b0 = (unit % FIN_GPQ) * FIN_G;
            if (b0 >= nb) return;  // uniform
            const int b1 = b0 + FIN_G < nb ? b0 + FIN_G : nb;
            first.has_lo = b0 > 0;
            first.lo = ends[0];
            first.hi = ends[b1 - b0];
            first.e0 = 1;
            first.e1 = 1 + (b1 - b0);
        } else {
            // The union's ranges follow the bucket ends of all its queues
            // merged, up to the reference bound: a range between consecutive
            // merged ends holds at most one bucket's worth of each queue,
            // wherever each queue's keys lie.  Union workgroup g takes
            // consecutive merged ends g S .. g S + S - 1, S = ceil(M / FIN_NU).
            unsigned long long *mend = st1, *mer = st2;  // [queue][SAE_NBUCKET], merged
            __shared__ uint32_t mcnt[SAE_MAX_QUEUES], mtot;
            const unsigned long long rb = f.thr[rq];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int i = tid + h * FIN_THREADS, qq = i / SAE_NBUCKET, j = i % SAE_NBUCKET;
                const bool ok = qq < Q && ((src >> qq) & 1u) && j < f.nb[qq];
                mend[i] = ok ? uend[h] : ~0ull;  // ascending per queue, unused slots last
            }
            lds_barrier();
            if (tid < SAE_MAX_QUEUES) {  // each queue's ends at or below the reference bound
                const int nq = (tid < Q && ((src >> tid) & 1u)) ? f.nb[tid] : 0;
                const unsigned long long *eq = mend + tid * SAE_NBUCKET;
                int l = 0;
#pragma unroll
                for (int st = SAE_NBUCKET; st > 0; st >>= 1)
                    if (l + st <= nq && eq[l + st - 1] <= rb) l += st;
                mcnt[tid] = (uint32_t)l;
            }
            lds_barrier();
            if (tid == 0) {
                uint32_t m = 0;
                for (int qq = 0; qq < SAE_MAX_QUEUES; ++qq) m += mcnt[qq];
                mtot = m;
            }
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int i = tid + h * FIN_THREADS, qq = i / SAE_NBUCKET, j = i % SAE_NBUCKET;
                if ((uint32_t)j < mcnt[qq]) {
                    // rank in the merge, equal ends ordered by queue
                    const unsigned long long v = mend[i];
                    uint32_t r = (uint32_t)j;
                    for (int q2 = 0; q2 < SAE_MAX_QUEUES; ++q2) {
                        if (q2 == qq || mcnt[q2] == 0) continue;
                        const unsigned long long *e2 = mend + q2 * SAE_NBUCKET;
                        const int n2 = (int)mcnt[q2];
                        int l = 0;
#pragma unroll
                        for (int st = SAE_NBUCKET; st > 0; st >>= 1)
                            if (l + st <= n2 && (q2 < qq ? e2[l + st - 1] <= v : e2[l + st - 1] < v)) l += st;
                        r += (uint32_t)l;
                    }
                    mer[r] = v;
                }
            }
            lds_barrier();
            const uint32_t M = mtot;
            const uint32_t S = (M + FIN_NU - 1) / FIN_NU;
            const uint32_t g = (uint32_t)(unit - n_group);
            const uint32_t r0 = g * S;
            if (r0 >= M) return;  // uniform
            const uint32_t r1 = r0 + S < M ? r0 + S : M;
            const uint32_t cnt = r1 - r0;
            const uint32_t stride = (cnt + FIN_G - 1) / FIN_G;
            const int nbk = (int)((cnt + stride - 1) / stride);
            if (tid == 0) ends[0] = r0 > 0 ? mer[r0 - 1] : 0ull;
            if (tid < nbk) {
                const uint32_t pos = r0 + (uint32_t)(tid + 1) * stride - 1;
                ends[1 + tid] = mer[pos < r1 ? pos : r1 - 1];
            }
            lds_barrier();
            first.has_lo = r0 > 0;
            first.lo = ends[0];
            first.hi = ends[nbk];
            first.e0 = 1;
            first.e1 = 1 + nbk;
        }
        const long long ob = ((long long)inst * Q + q) * c.max_k;
        const bool is_ef = group && q == c.ef_queue;
        const int n1 = f.n1;
        auto out = [&](uint32_t rank, unsigned long long e) {
            const int32_t id = (int32_t)(uint32_t)(e & 0xFFFFFFFFull);
            if (group) {
                a.victims[ob + rank] = id;
                if (a.scores) a.scores[ob + rank] = __uint_as_float((uint32_t)(e >> 32));
                c.sel[ob + rank] = e;
                if (is_ef) dec[rank] = id;
            } else {
                dec[n1 + (int)rank] = id;
            }
        };
        fin_rank(c, inst, f, src, ends, first, need, st1, st2, out);
        return;
    }
    // the finisher
    if (!f.any_fail) {
        if (tid < Q) {
            const long long iq = (long long)inst * Q + tid;
            a.count[iq] = (int32_t)f.need[tid];
            c.sel_count[iq] = (int32_t)f.need[tid];
            uint32_t *dbg = c.sel_stats + iq * 4;
            dbg[0] = (f.thr[tid] == ~0ull) ? f.C[tid] : 0xFFFFFFFFu;
            dbg[1] = f.C[tid];
            dbg[2] = f.over[tid];
            dbg[3] = 0;
        }
        if (tid == 0) {
            a.decision_count[inst] = f.d;
            // a cascading decision is completed (and counted) by k_cascade
            if (!(a.flags & SAE_SS_CASCADE)) commit_bookkeeping(c.state[inst], f.d, (a.flags & SAE_SS_COMMIT) != 0);
        }
        return;
    }
    fin_exact(c, a, inst, kq, f, P, lds_bytes, fdyn);
}

// ---------------------------------------------------------------------------
// Batched engine: one workgroup per instance (N <= 65,536 blocks).  Per
// queue, composite e = key << 16 | id (48 bits, distinct).
//  * The first pass reads the pool once, scores every evictable block (Eq.
//    1-3) and caches its key and queue (5 B per block) for the later passes,
//    counts each queue's evictable blocks and histograms the top digit of e;
//    need = min(k, evictable).  A queue whose need is all of its blocks takes
//    them all; otherwise the bin holding its need-th element gives a range
//    [lo, hi) of e: every element below lo is selected, and `rem` more from
//    inside the range.  When the range holds exactly `rem` elements, every
//    element below hi is selected.
//  * While the open ranges hold more elements than the candidate buffer, a
//    pass over the cached keys histograms the next digit inside each range
//    (equal keys spread on the id digits).
//  * The collect pass appends every selected element below lo to its queue's
//    list and every element inside the range to the candidate buffer; a
//    candidate is selected when fewer than `rem` candidates of its queue are
//    smaller, and goes straight to list position below + its rank.
//  * Each queue's list (at most max_k elements) is sorted, written out, and
//    the decision merged from the lists (Algorithm 1).
#define BATCH_CAND 2048  // candidate elements beyond the largest lists in LDS
#define BATCH_LQ 128     // blocks a wave's scoring list holds: < 64 left + 64 pushed
#define BATCH_LQ_BYTES (SEL_THREADS / SAE_WAVE * 2 * 3 * BATCH_LQ * 4)  // the first pass's lists (48 KiB)
struct BatchSel {
    unsigned long long lo[SAE_MAX_QUEUES], hi[SAE_MAX_QUEUES];
    uint32_t nev[SAE_MAX_QUEUES], need[SAE_MAX_QUEUES], rem[SAE_MAX_QUEUES], remv[SAE_MAX_QUEUES];
    uint32_t lcnt[SAE_MAX_QUEUES], ccnt[SAE_MAX_QUEUES], coff[SAE_MAX_QUEUES];
    int32_t mode[SAE_MAX_QUEUES];  // 0: none, 1: all, 2: below lo plus rem from [lo, hi), 3: below hi
    int32_t active[SAE_MAX_QUEUES];
    int32_t sh[SAE_MAX_QUEUES], w[SAE_MAX_QUEUES];  // the next digit: bits sh .. sh + w - 1 of e
    uint32_t mn[SAE_MAX_QUEUES], mx[SAE_MAX_QUEUES];  // smallest and largest key
    Crossing cr[SAE_MAX_QUEUES];
    uint32_t seg_tot[16];
    uint32_t open_cnt, st;
    int32_t pe;
};

// A pass over the cached keys of one instance: fn(q, e) for every evictable
// block, 8 blocks per thread loaded together.
template <typename Fn>
__device__ __forceinline__ void batch_cached_pass(const DevCtx &c, int inst, Fn fn)
{
    const int N = c.N, tid = threadIdx.x;
    const long long base = (long long)inst * N;
    if ((N & 3) == 0) {
        // four consecutive blocks per thread and load (16 bytes of keys, 4 of
        // queues), four such groups in flight: a quarter of the load
        // instructions of one block per lane
        const int ng = N / 4;  // groups of four blocks
        const uint4 *k4 = reinterpret_cast<const uint4 *>(c.bkey + base);
        const uint32_t *q4 = reinterpret_cast<const uint32_t *>(c.bq + base);
        for (int g0 = 0; g0 < ng; g0 += 4 * SEL_THREADS) {
            uint4 kv[4];
            uint32_t qv[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int gi = g0 + u * SEL_THREADS + tid;
                const bool in = gi < ng;
                kv[u] = k4[in ? gi : 0];  // clamped: every load unconditional, in flight together
                qv[u] = q4[in ? gi : 0];
                qv[u] = in ? qv[u] : 0u;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const uint32_t b0 = (uint32_t)(g0 + u * SEL_THREADS + tid) * 4u;
                const uint32_t kk[4] = {kv[u].x, kv[u].y, kv[u].z, kv[u].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t qb = (qv[u] >> (8 * e)) & 0xFFu;
                    if (qb) fn((int)qb - 1, ((unsigned long long)kk[e] << 16) | (b0 + (uint32_t)e));
                }
            }
        }
        return;
    }
    const int nj = (N + SEL_THREADS - 1) / SEL_THREADS;
    for (int j0 = 0; j0 < nj; j0 += 8) {
        uint32_t kv[8], qv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int b = tid + (j0 + u) * SEL_THREADS;
            const bool in = (j0 + u) < nj && b < N;
            const long long g = base + (in ? b : 0);
            kv[u] = c.bkey[g];
            qv[u] = in ? (uint32_t)c.bq[g] : 0u;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (qv[u]) fn((int)qv[u] - 1, ((unsigned long long)kv[u] << 16) | (uint32_t)(tid + (j0 + u) * SEL_THREADS));
    }
}

// After a histogram of every open queue's digit over its range: narrow the
// range to the crossing bin, and move to the next digit below it.
__device__ void batch_narrow(BatchSel &bs, int Q)
{
    const int tid = threadIdx.x;
    if (tid < Q && bs.active[tid]) {
        const Crossing cr = bs.cr[tid];
        const int sh = bs.sh[tid];
        const unsigned long long lo = bs.lo[tid] + ((unsigned long long)cr.bin << sh);
        bs.lo[tid] = lo;
        bs.hi[tid] = lo + (1ull << sh);
        bs.rem[tid] -= cr.below;
        bs.ccnt[tid] = cr.cnt;
        if (cr.cnt == bs.rem[tid] || sh == 0) {  // the whole bin is selected (a single value when sh = 0)
            bs.mode[tid] = 3;
            bs.active[tid] = 0;
            bs.ccnt[tid] = 0;
        } else {
            const int w = sh < SAE_DIGIT_BITS ? sh : SAE_DIGIT_BITS;
            bs.w[tid] = w;
            bs.sh[tid] = sh - w;
        }
    }
    lds_barrier();
    if (tid == 0) {
        uint32_t n = 0;
        for (int q = 0; q < Q; ++q) n += bs.active[q] ? bs.ccnt[q] : 0u;
        bs.open_cnt = n;
    }
    lds_barrier();
}

__global__ void __launch_bounds__(SEL_THREADS) k_batched(DevCtx c, SelectArgs a, int P, int dyn_elems)
{
    extern __shared__ unsigned long long sh_dyn[];  // hist [Q][SAE_BINS] u32, later lists [Q][Pe] + candidates
    uint32_t *hist = reinterpret_cast<uint32_t *>(sh_dyn);
    unsigned long long *lists = sh_dyn;
    __shared__ BatchSel bs;
    __shared__ ScoreTab tab;
    __shared__ int32_t cnt_s[SAE_MAX_QUEUES];
    const int inst = blockIdx.x;
    const int Q = c.Q, N = c.N;
    const int tid = threadIdx.x, lane = lane_id();
    const long long base = (long long)inst * N;
    load_score_tab(tab, c.state[inst], c);
    if (tid < SAE_MAX_QUEUES) {
        bs.nev[tid] = 0;
        bs.lcnt[tid] = 0;
        bs.active[tid] = 0;
        bs.mode[tid] = 0;
        bs.ccnt[tid] = 0;
        bs.mn[tid] = 0xFFFFFFFFu;
        bs.mx[tid] = 0;
    }
    if (tid == 0) bs.st = 0;
    lds_barrier();

    // first pass: score, cache, count, smallest and largest key per queue
    uint32_t cnt_r[SAE_MAX_QUEUES], mn_r[SAE_MAX_QUEUES], mx_r[SAE_MAX_QUEUES];
#pragma unroll
    for (int q = 0; q < SAE_MAX_QUEUES; ++q) {
        cnt_r[q] = 0;
        mn_r[q] = 0xFFFFFFFFu;
        mx_r[q] = 0;
    }
    uint32_t st = 0;
    {
        // A wave's lanes hold blocks of every queue kind, and Eq. 1 (ln,
        // erfc) and Eq. 2 are long: scored in place, every wave would run
        // both.  So the blocks of log-normal and structural queues are queued
        // per wave in LDS with their fields (the dynamic LDS is free until
        // the digit passes) and scored 64 at a time, one kind per wave-wide
        // step; the other kinds cost a few operations and are scored in place.
        // The next step's loads go out before this step is scored.
        uint32_t *wq = reinterpret_cast<uint32_t *>(sh_dyn) + (tid / SAE_WAVE) * 2 * 3 * BATCH_LQ;
        uint32_t nq0 = 0, nq1 = 0;  // fill of the log-normal and structural lists (wave-uniform)
        const unsigned long long lt = lanemask_lt();
        // the queues of each list's kind and of the kinds scored in place
        // (bit q): a block's counts only touch those
        uint32_t qm_ln = 0, qm_st = 0;
        for (int qq = 0; qq < Q; ++qq) {
            qm_ln |= (tab.kind[qq] == SAE_KIND_LOGNORMAL) ? 1u << qq : 0u;
            qm_st |= (tab.kind[qq] == SAE_KIND_STRUCTURAL) ? 1u << qq : 0u;
        }
        const uint32_t qm_rest = ((1u << Q) - 1u) & ~(qm_ln | qm_st);
        auto finish = [&](int b, uint32_t m, uint32_t key, bool ev, uint32_t qmask) {
            const int q = meta_queue(m);
            if (ev) {
#pragma unroll
                for (int qq = 0; qq < SAE_MAX_QUEUES; ++qq) {
                    if (qq >= Q) break;  // uniform
                    if (!((qmask >> qq) & 1u)) continue;  // uniform
                    cnt_r[qq] += (qq == q) ? 1u : 0u;
                    mn_r[qq] = (qq == q) ? min(mn_r[qq], key) : mn_r[qq];
                    mx_r[qq] = (qq == q) ? max(mx_r[qq], key) : mx_r[qq];
                }
            }
            c.bkey[base + b] = key;
            c.bq[base + b] = ev ? (uint8_t)(q + 1) : (uint8_t)0;
        };
        // Score the lists: each one that holds 64 (or, at the end, whatever
        // it holds).  One call site, so that the two long key functions are
        // compiled once.
        auto drain = [&](bool final) {
#pragma unroll 1
            for (int which = 0; which < 2; ++which) {
                uint32_t &nq = which == 0 ? nq0 : nq1;
                const uint32_t n = final ? nq : (nq >= SAE_WAVE ? (uint32_t)SAE_WAVE : 0u);
                if (n == 0) continue;  // uniform
                nq -= n;
                const uint32_t *w = wq + which * 3 * BATCH_LQ;
                const bool act = (uint32_t)lane < n;
                const uint32_t p = nq + (act ? (uint32_t)lane : 0u);
                const int32_t la = (int32_t)w[p];
                const uint32_t off = w[BATCH_LQ + p], mb = w[2 * BATCH_LQ + p];
                const uint32_t m = mb & 0xFFFFu;
                if (act) {
                    const uint32_t key = which == 0 ? key_lognormal(a.now, la, m, tab, st)
                                                    : key_structural(a.now, la, m, off, tab, st);
                    finish((int)(mb >> 16), m, key, true, which == 0 ? qm_ln : qm_st);
                }
            }
        };
        // Each lane takes blocks tid + 1024 j (consecutive lanes, consecutive
        // blocks: coalesced loads and key-cache stores), four j per step; the
        // next step's loads are issued before this step is scored (indices
        // past the pool load block 0).
        const int nj = (N + SEL_THREADS - 1) / SEL_THREADS;
        auto ld = [&](int j0, int32_t (&l)[4], uint32_t (&mm)[4], uint32_t (&o)[4]) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int b = tid + (j0 + u) * SEL_THREADS;
                const long long g = base + (((j0 + u) < nj && b < N) ? b : 0);
                l[u] = c.la[g];
                mm[u] = c.meta[g];
                o[u] = c.off[g];
            }
        };
        int32_t lc[4], ln[4];
        uint32_t mc[4], mn2[4], oc[4], on[4];
        ld(0, lc, mc, oc);
        for (int j0 = 0; j0 < nj; j0 += 4) {  // uniform
            ld(j0 + 4, ln, mn2, on);
#pragma unroll 1
            for (int e = 0; e < 4; ++e) {
                // one block per lane: scored in place, or queued
                const int b = tid + (j0 + e) * SEL_THREADS;
                const bool in = (j0 + e) < nj && b < N;
                const int32_t la = e == 0 ? lc[0] : (e == 1 ? lc[1] : (e == 2 ? lc[2] : lc[3]));
                const uint32_t off = e == 0 ? oc[0] : (e == 1 ? oc[1] : (e == 2 ? oc[2] : oc[3]));
                const uint32_t m = e == 0 ? mc[0] : (e == 1 ? mc[1] : (e == 2 ? mc[2] : mc[3]));
                const bool ev = in && meta_evictable(m) && meta_queue(m) < Q;
                const int kind = ev ? tab.kind[meta_queue(m)] : -1;
                const bool to0 = kind == SAE_KIND_LOGNORMAL, to1 = kind == SAE_KIND_STRUCTURAL;
                if (in && !to0 && !to1) finish(b, m, ev ? key_cheap(kind, a.now, la, m, tab, st) : 0u, ev, qm_rest);
                const unsigned long long m0 = __ballot(to0), m1 = __ballot(to1);
                if (to0 || to1) {
                    const uint32_t p = to0 ? nq0 + (uint32_t)__popcll(m0 & lt) : nq1 + (uint32_t)__popcll(m1 & lt);
                    uint32_t *w = wq + (to0 ? 0 : 3 * BATCH_LQ);
                    w[p] = (uint32_t)la;
                    w[BATCH_LQ + p] = off;
                    w[2 * BATCH_LQ + p] = m | ((uint32_t)b << 16);
                }
                nq0 += (uint32_t)__popcll(m0);
                nq1 += (uint32_t)__popcll(m1);
                __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
                __builtin_amdgcn_wave_barrier();
                drain(false);
                __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
                __builtin_amdgcn_wave_barrier();
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                lc[u] = ln[u];
                mc[u] = mn2[u];
                oc[u] = on[u];
            }
        }
        drain(true);  // what the lists still hold
    }
#pragma unroll
    for (int q = 0; q < SAE_MAX_QUEUES; ++q) {
        uint32_t v = cnt_r[q], lo = mn_r[q], hi = mx_r[q];
        for (int o = 32; o > 0; o >>= 1) {
            v += __shfl_xor(v, o, SAE_WAVE);
            lo = min(lo, (uint32_t)__shfl_xor(lo, o, SAE_WAVE));
            hi = max(hi, (uint32_t)__shfl_xor(hi, o, SAE_WAVE));
        }
        if (lane == 0 && v) {
            atomicAdd(&bs.nev[q], v);
            atomicMin(&bs.mn[q], lo);
            atomicMax(&bs.mx[q], hi);
        }
    }
    lds_barrier();
    if (tid < Q) {
        const int kk = inst_k(a, inst, c.max_k);
        const uint32_t need = (uint32_t)min((long long)kk, (long long)bs.nev[tid]);
        bs.need[tid] = need;
        bs.rem[tid] = need;
        if (need == 0) bs.mode[tid] = 0;
        else if (need >= bs.nev[tid]) bs.mode[tid] = 1;
        else {
            // the first digit: the highest bits where the queue's keys differ,
            // or the id bits when every key is equal
            const uint32_t kx = bs.mn[tid] ^ bs.mx[tid];
            const int top = kx ? 16 + (32 - __clz(kx)) : 16;  // bits of e below the common prefix
            const unsigned long long mn = (unsigned long long)bs.mn[tid] << 16;
            const int w = top < SAE_DIGIT_BITS ? top : SAE_DIGIT_BITS;
            bs.w[tid] = w;
            bs.sh[tid] = top - w;
            bs.lo[tid] = (mn >> top) << top;
            bs.hi[tid] = bs.lo[tid] + (1ull << top);
            bs.ccnt[tid] = bs.nev[tid];
            bs.mode[tid] = 2;
            bs.active[tid] = 1;
        }
    }
    lds_barrier();
    if (tid == 0) {  // list segments of Pe = pow2 >= the largest need
        uint32_t mx = 1;
        for (int q = 0; q < Q; ++q) mx = bs.need[q] > mx ? bs.need[q] : mx;
        bs.pe = pow2_ge((int)mx) < P ? pow2_ge((int)mx) : P;
    }
    lds_barrier();
    if (tid == 0) {
        uint32_t n = 0;
        for (int q = 0; q < Q; ++q) n += bs.active[q] ? bs.ccnt[q] : 0u;
        bs.open_cnt = n;
    }
    const int Pe = bs.pe;
    // the lists take Q x Pe elements at the start of the dynamic LDS, the
    // candidates follow (ranked by comparison, so their number is bounded)
    unsigned long long *cand = sh_dyn + (long long)Q * Pe;
    // every thread's cached keys are visible to the whole workgroup from here
    __syncthreads();
    // digit passes over the cached keys while the open ranges hold more than
    // the candidate buffer (each narrows every open range by up to 11 bits;
    // 48-bit composites need at most 5)
    for (int lev = 0; lev < 5 && bs.open_cnt > BATCH_CAND; ++lev) {  // uniform
        for (int i = tid; i < Q * SAE_BINS; i += blockDim.x) hist[i] = 0;
        if (tid < Q) bs.remv[tid] = bs.rem[tid];
        lds_barrier();
        batch_cached_pass(c, inst, [&](int q, unsigned long long e) {
            if (bs.active[q] && e >= bs.lo[q] && e < bs.hi[q])
                atomicAdd(&hist[q * SAE_BINS + ((uint32_t)(e >> bs.sh[q]) & ((1u << bs.w[q]) - 1u))], 1u);
        });
        lds_barrier();
        find_crossing(hist, Q, bs.remv, bs.active, bs.cr, bs.seg_tot);
        batch_narrow(bs, Q);
    }
    // candidates per open queue
    if (tid == 0) {
        uint32_t o = 0;
        for (int q = 0; q < Q; ++q) {
            bs.coff[q] = o;
            o += (bs.mode[q] == 2) ? bs.ccnt[q] : 0u;
        }
    }
    for (int i = tid; i < Q * Pe; i += blockDim.x) lists[i] = ~0ull;
    if (tid < Q) bs.ccnt[tid] = 0;  // from here the fill count of the queue's candidates
    lds_barrier();
    // collect
    batch_cached_pass(c, inst, [&](int q, unsigned long long e) {
        const int md = bs.mode[q];
        const bool sel = md == 1 || (md == 3 && e < bs.hi[q]) || (md == 2 && e < bs.lo[q]);
        const unsigned long long v = ((e >> 16) << 32) | (e & 0xFFFFull);
        if (sel) lists[(long long)q * Pe + atomicAdd(&bs.lcnt[q], 1u)] = v;
        else if (md == 2 && e < bs.hi[q]) cand[bs.coff[q] + atomicAdd(&bs.ccnt[q], 1u)] = v;
    });
    lds_barrier();
    // candidates: ranked among their queue's candidates, the first rem join the list
    {
        uint32_t tot = 0;
        for (int q = 0; q < Q; ++q) tot += (bs.mode[q] == 2) ? bs.ccnt[q] : 0u;
        for (uint32_t i = tid; i < tot; i += blockDim.x) {
            int q = 0;  // the queue whose candidates hold position i
            for (int qq = 0; qq < Q; ++qq)
                if (bs.mode[qq] == 2 && i >= bs.coff[qq] && i < bs.coff[qq] + bs.ccnt[qq]) q = qq;
            const unsigned long long v = cand[i];
            const uint32_t lo = bs.coff[q], n = bs.ccnt[q];
            uint32_t rk = 0;
            for (uint32_t t = 0; t < n; ++t) rk += (cand[lo + t] < v) ? 1u : 0u;
            if (rk < bs.rem[q]) lists[(long long)q * Pe + (bs.need[q] - bs.rem[q]) + rk] = v;
        }
    }
    if (st) atomicOr(&bs.st, st);
    lds_barrier();
    if (Pe >= 256 && 2 * Q * Pe <= dyn_elems) sort_segments_lds(lists, Q * Pe, Pe);
    else bitonic_sort_segments(lists, Q, Pe, Pe);
    if (tid < Q) cnt_s[tid] = (int32_t)min(bs.need[tid], (uint32_t)P);
    lds_barrier();
    for (int q = 0; q < Q; ++q) {
        const long long ob = ((long long)inst * Q + q) * c.max_k;
        for (int j = tid; j < cnt_s[q]; j += blockDim.x) {
            const unsigned long long e = lists[(long long)q * Pe + j];
            a.victims[ob + j] = (int32_t)(uint32_t)(e & 0xFFFFFFFFull);
            if (a.scores) a.scores[ob + j] = __uint_as_float((uint32_t)(e >> 32));
            c.sel[ob + j] = e;
        }
    }
    if (tid < Q) {
        a.count[(long long)inst * Q + tid] = cnt_s[tid];
        c.sel_count[(long long)inst * Q + tid] = cnt_s[tid];
    }
    const int kk = inst_k(a, inst, c.max_k);
    const int d = merge_decision(lists, Pe, cnt_s, Q, c.ef_queue, kk, a.decision + (long long)inst * c.max_k);
    if (tid == 0) {
        a.decision_count[inst] = d;
        if (!(a.flags & SAE_SS_CASCADE)) commit_bookkeeping(c.state[inst], d, (a.flags & SAE_SS_COMMIT) != 0);
        set_status(c.status, bs.st);
    }
}

// Kernels whose dynamic LDS may exceed 64 KiB ask for it explicitly, once per
// kernel and size (the attribute call costs host time on every launch otherwise).
hipError_t allow_lds(const void *fn, size_t bytes)
{
    if (bytes <= 64 * 1024) return hipSuccess;
    static thread_local const void *done_fn[16];
    static thread_local size_t done_bytes[16];
    for (int i = 0; i < 16; ++i)
        if (done_fn[i] == fn && done_bytes[i] >= bytes) return hipSuccess;
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess) return e;
    for (int i = 0; i < 16; ++i)
        if (done_fn[i] == nullptr || done_fn[i] == fn) {
            done_fn[i] = fn;
            done_bytes[i] = bytes;
            break;
        }
    return hipSuccess;
}

int pow2_at_least(int x)
{
    int p = 1;
    while (p < x) p <<= 1;
    return p;
}

// ---------------------------------------------------------------------------
// Cascading decision (SAE_SS_CASCADE): k successive Evict() calls of
// Algorithm 1 on the live state, where a parent whose last cached child is
// taken becomes a leaf for the next call.  With kappa(b) = (stage, key, id)
// (stage 0 for the evict-first queue, keyed by num_tokens), a block can be
// taken once every cached child has been, and the calls take blocks in the
// order of E(b) = max(kappa(b), E(children)), equal E (one path of the tree)
// child first.  Every block among the first k has E at most kappa of the
// snapshot decision's k-th victim, so all of them are reached from that
// decision by walking up parents: round r takes the blocks added in round
// r - 1 (round 0: the snapshot decision, sorted by kappa), counts them
// towards their parents (global counters, reset afterwards) and adds a parent
// when its last cached child arrives, with E = max(kappa(parent), the largest
// E of its children) and round r + 1 (which orders equal E child first).  The
// new blocks are sorted and merged into the sorted candidates, which keep
// only the first k.  Round 0 (up to k blocks) and the E of the parents it
// completes run over many workgroups (k_casc_round0, k_casc_parents); the
// later rounds, whose frontiers are small, in one workgroup of 1024 threads
// per instance (k_cascade).  The per-block counters come in two sets that
// calls alternate between; round 0 also zeroes the entries the previous call
// left in the other set, so they are clean when the call after uses them.
constexpr int CASC_THREADS = 1024;
constexpr int CASC_PER = 4;  // candidates per thread: k <= CASC_THREADS * CASC_PER
constexpr int CASC0_THREADS = 64;

struct CascEl {
    unsigned long long e;  // E (stage << 56 | key << 24 | id of the block that sets it)
    uint32_t id, rnd;
};

__device__ __forceinline__ bool casc_less(const CascEl &a, const CascEl &b)
{
    return a.e < b.e || (a.e == b.e && a.rnd < b.rnd);
}

__device__ __forceinline__ unsigned long long casc_kappa_of(const ScoreTab &tab, int32_t now, uint32_t b, uint32_t m,
                                                            int32_t la, uint32_t off, uint32_t &st)
{
    const uint32_t key = block_key(now, la, m, off, tab, st);
    const unsigned long long stage = (tab.kind[meta_queue(m)] == SAE_KIND_EVICT_FIRST) ? 0ull : 1ull;
    return (stage << 56) | ((unsigned long long)key << 24) | (unsigned long long)(b & 0xFFFFFFu);
}

__device__ __forceinline__ unsigned long long casc_kappa(const DevCtx &c, const ScoreTab &tab, int32_t now,
                                                         long long base, uint32_t b, uint32_t &st)
{
    return casc_kappa_of(tab, now, b, c.meta[base + b], c.la[base + b], c.off[base + b], st);
}

// number of elements of the sorted x[0..n) below v
__device__ __forceinline__ int casc_rank(const CascEl *x, int n, const CascEl &v)
{
    int lo = 0, hi = n;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (casc_less(x[mid], v)) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

// Round 0: one thread per snapshot victim records its kappa, raises its
// parent's largest E and counts itself towards the parent; the victim that
// completes a parent's count of cached children lists the parent if it is
// valid and unreferenced.  Listing needs only the count, and k_cascade reads
// the maxima after this launch has ended, so no ordering between the
// workgroups (and the XCDs they run on) is needed.
__global__ void __launch_bounds__(CASC0_THREADS) k_casc_round0(DevCtx c, SelectArgs a)
{
    __shared__ ScoreTab tab;
    const int inst = blockIdx.y;
    const long long base = (long long)inst * c.N;
    load_score_tab(tab, c.state[inst], c);
    {
        // zero what the previous call left in the other set: its touched
        // blocks, or every block when its list overflowed
        const int nt = c.casc_nt_prev[inst];
        const long long stride = (long long)gridDim.x * CASC0_THREADS;
        const long long i0 = (long long)blockIdx.x * CASC0_THREADS + threadIdx.x;
        if (nt <= c.casc_tl) {
            const int32_t *touch = c.casc_touch_prev + (long long)inst * c.casc_tl;
            for (long long i = i0; i < nt; i += stride) {
                const int32_t p = touch[i];
                c.casc_cnt_prev[base + p] = 0;
                c.casc_e_prev[base + p] = 0ull;
            }
        } else {
            for (long long b = i0; b < c.N; b += stride) {
                c.casc_cnt_prev[base + b] = 0;
                c.casc_e_prev[base + b] = 0ull;
            }
        }
    }
    __syncthreads();
    const int j = blockIdx.x * CASC0_THREADS + threadIdx.x;
    if (j >= a.decision_count[inst]) return;
    const long long slot = (long long)inst * c.max_k + j;
    const uint32_t b = (uint32_t)a.decision[slot];
    const int32_t p = c.parent[base + b];
    uint32_t st = 0;
    const unsigned long long e = casc_kappa(c, tab, a.now, base, b, st);
    c.casc_k0[slot] = e;
    if (p >= 0 && p < c.N) {
        atomicMax(&c.casc_e[base + p], e);
        const int cc = c.child_count[base + p];
        const uint32_t pm = c.meta[base + p];
        const int old = atomicAdd(&c.casc_cnt[base + p], 1);
        int32_t *n = c.casc_n + 4 * inst;
        if (old == 0) {
            const int t = atomicAdd(&n[0], 1);
            if (t < c.casc_tl) c.casc_touch[(long long)inst * c.casc_tl + t] = p;
        }
        if (old + 1 == cc && (pm & (SAE_META_VALID | SAE_META_REF)) == SAE_META_VALID)
            c.casc_prom[(long long)inst * c.max_k + atomicAdd(&n[1], 1)] = p;
    }
    if (st) set_status(c.status, st);
}

// E of each parent that round 0 completed (every child's E is in: the
// previous launch has ended); the parents below the admission bound, the
// snapshot decision's k-th victim (none while it holds fewer than k), are
// listed with their E for k_cascade.  They enter round 1, so E equal to the
// bound does not pass.
__global__ void __launch_bounds__(CASC0_THREADS) k_casc_parents(DevCtx c, SelectArgs a)
{
    __shared__ ScoreTab tab;
    const int inst = blockIdx.y;
    const long long base = (long long)inst * c.N;
    load_score_tab(tab, c.state[inst], c);
    __syncthreads();
    const int i = blockIdx.x * CASC0_THREADS + threadIdx.x;
    if (i >= c.casc_n[4 * inst + 1]) return;
    const int k = inst_k(a, inst, c.max_k);
    const int d0 = a.decision_count[inst];
    const long long row = (long long)inst * c.max_k;
    const unsigned long long bound = (d0 >= k && k > 0) ? c.casc_k0[row + k - 1] : ~0ull;
    const uint32_t p = (uint32_t)c.casc_prom[row + i];
    uint32_t st = 0;
    const unsigned long long kp = casc_kappa(c, tab, a.now, base, p, st);
    const unsigned long long ec = c.casc_e[base + p];
    const unsigned long long e = kp > ec ? kp : ec;
    if (e < bound) {
        const int t = atomicAdd(&c.casc_n[4 * inst + 3], 1);
        c.casc_pe[row + t] = e;
        c.casc_aid[row + t] = (int32_t)p;
    }
    if (st) set_status(c.status, st);
}

__global__ void __launch_bounds__(CASC_THREADS) k_cascade(DevCtx c, SelectArgs a)
{
    extern __shared__ unsigned long long casc_lds[];
    const int kmax = c.max_k;
    CascEl *cur = reinterpret_cast<CascEl *>(casc_lds);  // [kmax] sorted candidates
    CascEl *nw = cur + kmax;                             // [pow2 >= kmax] the round's new blocks
    __shared__ ScoreTab tab;
    __shared__ int n_cur_s, n_new_s, n_touch_s, n_adm_s;
    __shared__ uint32_t st_s;
    const int inst = blockIdx.x;
    const int tid = threadIdx.x;
    const long long base = (long long)inst * c.N;
    const int k = inst_k(a, inst, kmax);
    int32_t *dec = a.decision + (long long)inst * kmax;
    int32_t *cnt = c.casc_cnt + base;
    unsigned long long *emax = c.casc_e + base;
    int32_t *touch = c.casc_touch + (long long)inst * c.casc_tl;
    const int32_t *adm = c.casc_aid + (long long)inst * kmax;
    const unsigned long long *adm_e = c.casc_pe + (long long)inst * kmax;
    const int d0 = a.decision_count[inst];
    load_score_tab(tab, c.state[inst], c);
    if (tid == 0) {
        n_cur_s = d0;
        n_touch_s = c.casc_n[4 * inst];
        n_adm_s = c.casc_n[4 * inst + 3];
        st_s = 0;
    }
    uint32_t st = 0;
    // the snapshot decision, already in kappa order
    for (int j = tid; j < d0; j += CASC_THREADS) {
        CascEl x;
        x.e = c.casc_k0[(long long)inst * kmax + j];
        x.id = (uint32_t)dec[j];
        x.rnd = 0;
        cur[j] = x;
    }
    __syncthreads();
    for (uint32_t r = 0;; ++r) {
        if (tid == 0) n_new_s = 0;
        __syncthreads();
        const int n_cur = n_cur_s;
        // admission bound: the k-th candidate so far (none while fewer than k)
        CascEl bound;
        bound.e = ~0ull;
        bound.rnd = 0xFFFFFFFFu;
        if (n_cur >= k && k > 0) bound = cur[k - 1];
        if (r == 0) {
            // the parents that round 0 completed, below the snapshot's bound
            const int n_adm = n_adm_s;
            for (int i = tid; i < n_adm; i += CASC_THREADS) {
                CascEl y;
                y.e = adm_e[i];
                y.id = (uint32_t)adm[i];
                y.rnd = 1;
                nw[i] = y;
            }
            if (tid == 0) n_new_s = n_adm;
        } else {
            // each thread's (up to CASC_PER) frontier blocks; once the parent
            // is known, its maximum, count and every field its kappa needs go
            // out together
            CascEl fx[CASC_PER];
            int32_t fp[CASC_PER];
#pragma unroll
            for (int u = 0; u < CASC_PER; ++u) {
                const int j = tid + u * CASC_THREADS;
                fx[u] = cur[j < n_cur ? j : 0];
                const bool f = j < n_cur && fx[u].rnd == r;
                const int32_t p = c.parent[base + (f ? fx[u].id : 0u)];  // unconditional: no wait per block
                fp[u] = (f && p >= 0 && p < c.N) ? p : -1;
            }
            int old[CASC_PER], cc[CASC_PER], pla[CASC_PER];
            uint32_t pm[CASC_PER], po[CASC_PER];
#pragma unroll
            for (int u = 0; u < CASC_PER; ++u) {
                old[u] = -2;
                if (fp[u] >= 0) {
                    const long long q = base + fp[u];
                    atomicMax(&emax[fp[u]], fx[u].e);
                    old[u] = atomicAdd(&cnt[fp[u]], 1);
                    cc[u] = c.child_count[q];
                    pm[u] = c.meta[q];
                    pla[u] = c.la[q];
                    po[u] = c.off[q];
                }
            }
            // every maximum of this round is performed (in the one L2 this
            // workgroup's atomics go to) before any is read back below
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
            __syncthreads();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
#pragma unroll
            for (int u = 0; u < CASC_PER; ++u) {
                if (fp[u] < 0) continue;
                if (old[u] == 0) {
                    const int t = atomicAdd(&n_touch_s, 1);
                    if (t < c.casc_tl) touch[t] = fp[u];
                }
                // its last cached child, of a valid and unreferenced parent
                if (old[u] + 1 != cc[u] || (pm[u] & (SAE_META_VALID | SAE_META_REF)) != SAE_META_VALID) continue;
                const uint32_t p = (uint32_t)fp[u];
                CascEl y;
                const unsigned long long kp = casc_kappa_of(tab, a.now, p, pm[u], pla[u], po[u], st);
                const unsigned long long ec = __hip_atomic_load(&emax[p], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                y.e = kp > ec ? kp : ec;
                y.id = p;
                y.rnd = r + 1;
                if (!casc_less(y, bound)) continue;  // cannot be among the first k
                nw[atomicAdd(&n_new_s, 1)] = y;
            }
        }
        __syncthreads();
        const int n_new = n_new_s;
        if (n_new == 0) break;  // uniform
        // sort the new blocks (bitonic over the next power of two)
        int P = 1;
        while (P < n_new) P <<= 1;
        for (int j = n_new + tid; j < P; j += CASC_THREADS) {
            nw[j].e = ~0ull;
            nw[j].id = 0xFFFFFFFFu;
            nw[j].rnd = 0xFFFFFFFFu;
        }
        __syncthreads();
        for (int size = 2; size <= P; size <<= 1) {
            for (int stride = size >> 1; stride > 0; stride >>= 1) {
                for (int i = tid; i < P / 2; i += CASC_THREADS) {
                    const int lo = 2 * i - (i & (stride - 1));
                    const int hi = lo + stride;
                    const bool up = (lo & size) == 0;
                    const CascEl u = nw[lo], v = nw[hi];
                    if (casc_less(v, u) == up) {
                        nw[lo] = v;
                        nw[hi] = u;
                    }
                }
                __syncthreads();
            }
        }
        // merge by rank, everything read before anything is written; the
        // candidates below the smallest new block keep their places
        const int pos0 = casc_rank(cur, n_cur, nw[0]);
        CascEl xc[CASC_PER], xn[CASC_PER];
        int rc[CASC_PER], rn[CASC_PER];
#pragma unroll
        for (int u = 0; u < CASC_PER; ++u) {
            const int j = tid + u * CASC_THREADS;
            const int jc = pos0 + j;
            rc[u] = rn[u] = 0x7FFFFFFF;
            if (jc < n_cur) {
                xc[u] = cur[jc];
                rc[u] = jc + casc_rank(nw, n_new, xc[u]);
            }
            if (j < n_new) {
                xn[u] = nw[j];
                rn[u] = j + pos0 + casc_rank(cur + pos0, n_cur - pos0, xn[u]);
            }
        }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < CASC_PER; ++u) {
            if (rc[u] < k) cur[rc[u]] = xc[u];
            if (rn[u] < k) cur[rn[u]] = xn[u];
        }
        if (tid == 0) n_cur_s = min(k, n_cur + n_new);
        __syncthreads();
    }
    const int d = min(k, n_cur_s);
    for (int j = tid; j < d; j += CASC_THREADS) dec[j] = (int32_t)cur[j].id;
    // the per-block entries this call changed are zeroed by the next call's
    // round 0 (the other set is then in use)
    if (st) atomicOr(&st_s, st);
    __syncthreads();
    if (tid == 0) {
        c.casc_n[4 * inst] = 0;
        c.casc_n[4 * inst + 1] = 0;
        c.casc_nt[inst] = n_touch_s;
        c.casc_n[4 * inst + 3] = 0;
        a.decision_count[inst] = d;
        commit_bookkeeping(c.state[inst], d, (a.flags & SAE_SS_COMMIT) != 0);
        set_status(c.status, st_s);
    }
}

}  // namespace

bool batched_engine_fits(const DevCtx &c)
{
    if (c.N > BATCH_IPT * SEL_THREADS) return false;
    long long P = pow2_at_least(c.max_k);
    long long lds = (long long)c.Q * (P * 8 > SAE_BINS * 4 ? P * 8 : SAE_BINS * 4);
    return lds <= 128 * 1024;
}

hipError_t launch_select_scan(const DevCtx &c, const SelectArgs &a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1,
                              const PmArgs *pm, uint32_t *prep_calls)
{
    hipError_t e;
    const size_t lds_el = (size_t)LCAP * sizeof(unsigned long long);
    if (pm) {
        // steps 1 and 2 in the prefix match's launch, then its second pass
        if ((e = allow_lds((const void *)k_match_prep, lds_el)) != hipSuccess) return e;
        // one workgroup per compute unit (LDS): the prefix-match workgroups that fit beside the others take
        // the requests, up to 64 each
        const long long other = (long long)c.n_inst * (PREP_SAMPLE_WGS + c.Q);
        const long long avail = (long long)c.n_cu > other ? (long long)c.n_cu - other : 1;
        long long per = ((long long)pm->n_req + avail - 1) / avail;
        per = per < SEL_THREADS / SAE_WAVE ? SEL_THREADS / SAE_WAVE : (per > 64 ? 64 : per);
        const int n_pm = (int)(((long long)pm->n_req + per - 1) / per);
        const long long wgs = other + n_pm;
        const uint32_t calls = *prep_calls;
        hipLaunchKernelGGL(k_match_prep, dim3((unsigned)wgs), dim3(SEL_THREADS), lds_el, s, c, a, *pm,
                           (calls + 1u) * (uint32_t)PREP_SAMPLE_WGS, n_pm, (int)per);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        *prep_calls = calls + 1u;  // the sampling counters have moved on
        if (pm->flags & SAE_PM_INTERVALS) {
            e = launch_pm_place(c, pm->n_req, pm->max_len, pm->inst, pm->now, pm->flags, pm->matched_ids, s);
            if (e != hipSuccess) return e;
        }
    } else {
        // step 1: sample
        hipLaunchKernelGGL(k_sample, dim3(SAMPLE_WGS, c.n_inst), dim3(SCAN_THREADS), 0, s, c, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        // step 2: candidate bounds, bucket upper ends, the scan's filter entries
        if ((e = allow_lds((const void *)k_split, lds_el)) != hipSuccess) return e;
        hipLaunchKernelGGL(k_split, dim3(c.Q, c.n_inst), dim3(SEL_THREADS), lds_el, s, c, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    // step 3: streaming pass (with profiling, the events carry the dispatch's own start and end)
    if (ev0 && ev1)
        hipExtLaunchKernelGGL(k_scan, dim3(c.scan_gx, c.n_inst), dim3(SCAN_THREADS), 0, s, ev0, ev1, 0, c, a);
    else
        hipLaunchKernelGGL(k_scan, dim3(c.scan_gx, c.n_inst), dim3(SCAN_THREADS), 0, s, c, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // step 4: lists, decision and commit
    const int P = pow2_at_least(c.max_k);
    size_t lds = (size_t)2 * FIN_GCAP * sizeof(unsigned long long);  // staging of a range
    const size_t ex = (size_t)2 * (P < 256 ? 256 : P) * sizeof(unsigned long long);  // the exact path's sort
    if (ex > lds) lds = ex;
    if (lds < (size_t)SAE_BINS * sizeof(uint32_t)) lds = (size_t)SAE_BINS * sizeof(uint32_t);
    if ((e = allow_lds((const void *)k_final, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_final, dim3(c.Q * FIN_GPQ + FIN_NU + 1, c.n_inst), dim3(FIN_THREADS), lds, s, c, a, P,
                       (long long)lds);
    return hipGetLastError();
}

int scan_grid_x(int n_inst, int N)
{
    // 1024 workgroups of 4 waves over all instances (4 waves per SIMD), each
    // wave streaming several 256-block batches; no thread counts more than
    // 32768 evictable blocks
    long long want = ((long long)N + 4 * SCAN_BATCH - 1) / (4 * SCAN_BATCH);
    long long cap = 1024 / n_inst + 1;
    long long gx = want < cap ? want : cap;
    long long lo = ((long long)N + (long long)SCAN_THREADS * 32768 - 1) / ((long long)SCAN_THREADS * 32768);
    if (gx < lo) gx = lo;
    if (gx < 1) gx = 1;
    if (gx > 2048) gx = 2048;
    return (int)gx;
}

hipError_t launch_select_batched(const DevCtx &c, const SelectArgs &a, hipStream_t s)
{
    int P = pow2_at_least(c.max_k);
    // the histograms, then the lists and the candidate buffer
    const size_t h = (size_t)c.Q * SAE_BINS * 4, l = ((size_t)c.Q * P + BATCH_CAND) * 8;
    size_t lds = h > l ? h : l;
    if (lds < (size_t)BATCH_LQ_BYTES) lds = BATCH_LQ_BYTES;  // the first pass's scoring lists
    const int dyn_elems = (int)(lds / 8);
    hipError_t e = allow_lds((const void *)k_batched, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_batched, dim3(c.n_inst), dim3(SEL_THREADS), lds, s, c, a, P, dyn_elems);
    return hipGetLastError();
}

hipError_t launch_cascade(const DevCtx &c0, const SelectArgs &a, hipStream_t s, int set)
{
    // this call's counter set and the other one
    DevCtx c = c0;
    const long long nb = (long long)c0.n_inst * c0.N, nl = (long long)c0.n_inst * c0.casc_tl;
    const long long mine = set ? 1 : 0, other = 1 - mine;
    c.casc_cnt = c0.casc_cnt + mine * nb;
    c.casc_e = c0.casc_e + mine * nb;
    c.casc_touch = c0.casc_touch + mine * nl;
    c.casc_nt = c0.casc_nt + mine * c0.n_inst;
    c.casc_cnt_prev = c0.casc_cnt + other * nb;
    c.casc_e_prev = c0.casc_e + other * nb;
    c.casc_touch_prev = c0.casc_touch + other * nl;
    c.casc_nt_prev = c0.casc_nt + other * c0.n_inst;
    int P = 1;
    while (P < c.max_k) P <<= 1;
    const size_t lds = (size_t)(c.max_k + P) * sizeof(CascEl);
    hipError_t e = allow_lds((const void *)k_cascade, lds);
    if (e != hipSuccess) return e;
    const dim3 g0((c.max_k + CASC0_THREADS - 1) / CASC0_THREADS, c.n_inst);
    hipLaunchKernelGGL(k_casc_round0, g0, dim3(CASC0_THREADS), 0, s, c, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_casc_parents, g0, dim3(CASC0_THREADS), 0, s, c, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_cascade, dim3(c.n_inst), dim3(CASC_THREADS), lds, s, c, a);
    return hipGetLastError();
}
