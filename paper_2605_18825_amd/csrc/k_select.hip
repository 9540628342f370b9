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
#define SAMPLE_WGS SAE_SAMPLE_WGS
#define SAMPLE_CHUNK SAE_SAMPLE_CHUNK
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
// of two) stored back to back in LDS.  Index arithmetic by shifts and masks.
__device__ void bitonic_sort_segments(unsigned long long *a, int nseg, int P)
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
                unsigned long long *sg = a + ((long long)sgi << lp);
                const unsigned long long x = sg[lo], y = sg[hi];
                const bool up = ((lo >> lk) & 1) == 0;
                if ((x > y) == up) {
                    sg[lo] = y;
                    sg[hi] = x;
                }
            }
            __syncthreads();
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
    __syncthreads();
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
        __syncthreads();
        unsigned long long *t = src;
        src = dst;
        dst = t;
    }
    if (src != a) {
        for (int i = tid; i < P; i += blockDim.x) a[i] = src[i];
        __syncthreads();
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

// LDS working set of the per-(instance, queue) selection kernels.
#define LCAP 16384  // elements (128 KiB of LDS)

// Scratch for lds_select_bound (LDS).
struct BoundScratch {
    uint32_t hist[SAE_BINS];
    uint32_t rem[SAE_MAX_QUEUES];
    int32_t act[SAE_MAX_QUEUES];
    Crossing cr[SAE_MAX_QUEUES];
    uint32_t seg_tot[16];
    unsigned long long mn, mx;
};

// Among n distinct elements held in LDS, the bound B such that exactly `need`
// of them are <= B (1 <= need < n).  Radix select with 11-bit digits starting
// below the common prefix of the smallest and largest element, so a run of
// equal keys costs only the digits where the ids differ.  All threads call.
__device__ unsigned long long lds_select_bound(const unsigned long long *el, int n, uint32_t need, BoundScratch &b)
{
    const int tid = threadIdx.x;
    if (tid == 0) {
        b.mn = ~0ull;
        b.mx = 0;
    }
    __syncthreads();
    unsigned long long mn = ~0ull, mx = 0;
    for (int i = tid; i < n; i += blockDim.x) {
        unsigned long long e = el[i];
        mn = e < mn ? e : mn;
        mx = e > mx ? e : mx;
    }
    for (int d = 32; d > 0; d >>= 1) {
        unsigned long long o1 = __shfl_xor(mn, d, SAE_WAVE), o2 = __shfl_xor(mx, d, SAE_WAVE);
        mn = o1 < mn ? o1 : mn;
        mx = o2 > mx ? o2 : mx;
    }
    if (lane_id() == 0) {
        atomicMin(&b.mn, mn);
        atomicMax(&b.mx, mx);
    }
    __syncthreads();
    mn = b.mn;
    mx = b.mx;
    if (mn == mx) return mn;
    int sh = 64 - __clzll((long long)(mn ^ mx));
    unsigned long long prefix = mn >> sh;
    uint32_t rem = need;
    while (true) {
        const int w = sh < SAE_DIGIT_BITS ? sh : SAE_DIGIT_BITS;
        sh -= w;
        for (int i = tid; i < SAE_BINS; i += blockDim.x) b.hist[i] = 0;
        if (tid < SAE_MAX_QUEUES) {
            b.rem[tid] = (tid == 0) ? rem : 0u;
            b.act[tid] = (tid == 0);
        }
        __syncthreads();
        const uint32_t mask = (1u << w) - 1u;
        for (int i = tid; i < n; i += blockDim.x) {
            unsigned long long e = el[i];
            if ((sh + w >= 64) || (e >> (sh + w)) == prefix) atomicAdd(&b.hist[(uint32_t)(e >> sh) & mask], 1u);
        }
        __syncthreads();
        find_crossing(b.hist, 1, b.rem, b.act, b.cr, b.seg_tot);
        const Crossing c = b.cr[0];
        prefix = (prefix << w) | (unsigned long long)c.bin;
        const bool done = (c.cnt == rem) || (sh == 0);
        rem -= c.below;
        __syncthreads();
        if (done) break;
    }
    return (sh == 0) ? prefix : ((prefix << sh) | ((1ull << sh) - 1ull));
}

// ---------------------------------------------------------------------------
// Pool-scan engine, step 1: score a sample of every instance -- SAMPLE_WGS
// contiguous chunks spread evenly over the pool (the whole pool when it has
// at most SAMPLE_WGS * SAMPLE_CHUNK blocks) -- and record, per chunk, the
// (key << 32 | id) of every evictable sampled block with its queue, plus a
// per-queue histogram of the top 11 key bits (spread over SAE_HIST_STRIPES
// copies so that few workgroups add into the same counter).
__global__ void __launch_bounds__(SCAN_THREADS) k_sample(DevCtx c, SelectArgs a)
{
    extern __shared__ uint32_t sh_hist[];  // [Q][SAE_SBINS]
    __shared__ ScoreTab tab;
    __shared__ unsigned long long tmp[SAMPLE_CHUNK];
    __shared__ uint8_t tq[SAMPLE_CHUNK];
    __shared__ uint32_t qcnt[SAE_MAX_QUEUES], qoff[SAE_MAX_QUEUES], qfill[SAE_MAX_QUEUES];
    __shared__ uint32_t pos_s, st_s;
    const int inst = blockIdx.y;
    const int chunk = blockIdx.x;
    const int Q = c.Q;
    const long long N = c.N;
    const long long base = (long long)inst * N;
    load_score_tab(tab, c.state[inst], c);
    for (int i = threadIdx.x; i < Q * SAE_SBINS; i += blockDim.x) sh_hist[i] = 0;
    if (threadIdx.x < SAE_MAX_QUEUES) {
        qcnt[threadIdx.x] = 0;
        qfill[threadIdx.x] = 0;
    }
    if (threadIdx.x == 0) {
        pos_s = 0;
        st_s = 0;
    }
    __syncthreads();

    const bool whole = N <= (long long)SAMPLE_WGS * SAMPLE_CHUNK;
    const long long start = ((long long)chunk * N) / SAMPLE_WGS;
    const long long end = whole ? (((long long)chunk + 1) * N) / SAMPLE_WGS : start + SAMPLE_CHUNK;
    const long long reg = ((long long)inst * SAMPLE_WGS + chunk) * SAMPLE_CHUNK;
    uint32_t st = 0;
    for (long long b = start + threadIdx.x; b < end; b += blockDim.x) {
        const uint32_t m = c.meta[base + b];
        const int q = meta_queue(m);
        if (!meta_evictable(m) || q >= Q) continue;
        const uint32_t key = block_key(a.now, c.la[base + b], m, c.off[base + b], tab, st);
        atomicAdd(&sh_hist[q * SAE_SBINS + (key >> 23)], 1u);
        atomicAdd(&qcnt[q], 1u);
        const uint32_t p = atomicAdd(&pos_s, 1u);  // p < SAMPLE_CHUNK: one slot per sampled block
        tmp[p] = ((unsigned long long)key << 32) | (uint32_t)b;
        tq[p] = (uint8_t)q;
    }
    if (st) atomicOr(&st_s, st);
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t o = 0;
        for (int q = 0; q < SAE_MAX_QUEUES; ++q) {
            qoff[q] = o;
            o += qcnt[q];
        }
    }
    if (threadIdx.x < SAE_MAX_QUEUES)
        c.samp_qn[((long long)inst * SAMPLE_WGS + chunk) * SAE_MAX_QUEUES + threadIdx.x] = qcnt[threadIdx.x];
    __syncthreads();
    // the region holds queue 0's elements, then queue 1's, ...
    const uint32_t n = pos_s;
    for (uint32_t p = threadIdx.x; p < n; p += blockDim.x) {
        const int q = tq[p];
        const uint32_t pos = qoff[q] + atomicAdd(&qfill[q], 1u);
        c.samp[reg + pos] = tmp[p];
    }
    uint32_t *gh = c.shist + ((long long)inst * SAE_HIST_STRIPES + (chunk % SAE_HIST_STRIPES)) * Q * SAE_SBINS;
    for (int i = threadIdx.x; i < Q * SAE_SBINS; i += blockDim.x) {
        const uint32_t v = sh_hist[i];
        if (v) atomicAdd(&gh[i], v);
    }
    if (threadIdx.x == 0) set_status(c.status, st_s);
}

// Pool-scan engine, step 2: per (instance, queue), the candidate bound
// B = the r-th smallest sampled (key, id), r sized so that the pool holds
// about 1.5 need + a few standard deviations of blocks <= B.  The top key
// digit comes from the histogram; the rest from an exact select over the
// sampled elements of that bin, staged in LDS (a bin of equal keys --
// num_tokens of an evict-first queue, P = 0 of the last template blocks -- is
// split by block id).
__global__ void __launch_bounds__(SEL_THREADS) k_threshold(DevCtx c, SelectArgs a)
{
    extern __shared__ unsigned long long el[];  // [LCAP]
    __shared__ BoundScratch bs;
    __shared__ uint32_t qbase[SAMPLE_WGS], qpre[SAMPLE_WGS + 1], csum[SEL_THREADS / SAE_WAVE];
    __shared__ uint32_t tot_s, ns_s, bin_s, below_s;
    __shared__ unsigned long long bound_s;
    const int q = blockIdx.x;
    const int inst = blockIdx.y;
    const int Q = c.Q;
    const long long N = c.N;
    const int tid = threadIdx.x;
    if (tid == 0) {
        tot_s = 0;
        ns_s = 0;
        bound_s = ~0ull;
    }
    {
        // where queue q's elements start in each chunk's region, and how many
        uint32_t cnt = 0;
        if (tid < SAMPLE_WGS) {
            const uint32_t *qn = c.samp_qn + ((long long)inst * SAMPLE_WGS + tid) * SAE_MAX_QUEUES;
            uint32_t o = 0;
            for (int qq = 0; qq < q; ++qq) o += qn[qq];
            qbase[tid] = o;
            cnt = qn[q];
        }
        const uint32_t inc = wave_incl_scan(cnt);
        if (lane_id() == 63) csum[tid >> 6] = inc;
        __syncthreads();
        uint32_t pre = 0;
        for (int w = 0; w < (tid >> 6); ++w) pre += csum[w];
        if (tid < SAMPLE_WGS) qpre[tid] = pre + inc - cnt;
        if (tid == SAMPLE_WGS - 1) qpre[SAMPLE_WGS] = pre + inc;
    }
    __syncthreads();
    // histogram of the top 9 key bits over all stripes; thread t < 512 owns bin t
    uint32_t v = 0;
    if (tid < SAE_SBINS) {
#pragma unroll 8
        for (int st = 0; st < SAE_HIST_STRIPES; ++st) {
            uint32_t *g = c.shist + (((long long)inst * SAE_HIST_STRIPES + st) * Q + q) * SAE_SBINS + tid;
            v += *g;
            *g = 0;  // ready for the next call
        }
    }
    const uint32_t incl = wave_incl_scan(v);
    if (lane_id() == 63) csum[tid >> 6] = incl;
    __syncthreads();
    uint32_t pre = 0;
    for (int w = 0; w < (tid >> 6); ++w) pre += csum[w];
    const uint32_t cum = pre + incl;  // inclusive prefix over bins
    if (tid == SEL_THREADS - 1) tot_s = cum;
    __syncthreads();
    const uint32_t tot = tot_s;
    const long long S = (N <= (long long)SAMPLE_WGS * SAMPLE_CHUNK) ? N : (long long)SAMPLE_WGS * SAMPLE_CHUNK;
    const double f = (double)S / (double)N;
    const double est = (double)tot / f;
    const double need = fmin((double)inst_k(a, inst, c.max_k), est);
    const double nf = need * f;
    const uint32_t r = (uint32_t)ceil(nf * 1.25 + 3.0 * sqrt(nf) + 6.0);
    if (!(need > 0.0)) {
        if (tid == 0) bound_s = 0ull;
    } else if (est > 0.5 * (double)c.cand_cap && r < tot) {
        // the bin where the r-th sampled element lies
        if (tid < SAE_SBINS && cum - v < r && r <= cum) {
            bin_s = (uint32_t)tid;
            below_s = cum - v;
        }
        __syncthreads();
        const uint32_t bin = bin_s;
        const uint32_t rem = r - below_s;
        const unsigned long long edge = (((unsigned long long)bin + 1ull) << 55) - 1ull;
        // stage the sampled elements of queue q in that bin: index math first,
        // then every load in flight, then the LDS writes
        const unsigned long long *sp = c.samp + (long long)inst * SAMPLE_WGS * SAMPLE_CHUNK;
        const uint32_t nq = qpre[SAMPLE_WGS];
        for (uint32_t r0 = 0; r0 < nq; r0 += 16 * SEL_THREADS) {
            unsigned long long ev[16];
#pragma unroll
            for (int m = 0; m < 16; ++m) {
                const uint32_t i = r0 + tid + (uint32_t)m * SEL_THREADS;
                ev[m] = ~0ull;
                if (i < nq) {
                    int lo = 0, hi = SAMPLE_WGS - 1;  // last chunk with qpre <= i
                    while (lo < hi) {
                        const int mid = (lo + hi + 1) >> 1;
                        if (qpre[mid] <= i) lo = mid;
                        else hi = mid - 1;
                    }
                    ev[m] = sp[(long long)lo * SAMPLE_CHUNK + qbase[lo] + (i - qpre[lo])];
                }
            }
#pragma unroll
            for (int m = 0; m < 16; ++m) {
                if (ev[m] != ~0ull && (uint32_t)(ev[m] >> 55) == bin) {
                    const uint32_t pos = atomicAdd(&ns_s, 1u);
                    if (pos < LCAP) el[pos] = ev[m];
                }
            }
        }
        __syncthreads();
        const uint32_t ns = ns_s;
        unsigned long long bnd = edge;  // the whole bin
        if (rem < ns && ns <= LCAP) bnd = lds_select_bound(el, (int)ns, rem, bs);
        if (tid == 0) bound_s = bnd;
    }
    __syncthreads();
    if (tid == 0) c.thr[(long long)inst * Q + q] = bound_s;
}

// Pool-scan engine, step 3: one streaming pass over the whole pool.
// Each wave takes batches of SCAN_BATCH consecutive blocks: every lane loads
// 2 x 4 blocks with 16-, 8- and 16-byte loads (last_access, meta, off) into
// the wave's LDS staging area, the wave sorts the evictable blocks into three
// lists by queue kind (log-normal, structural, evict-first/recency) with
// ballots, and then scores each list with all lanes busy on the same code.
// Non-evictable blocks cost only their load and decode.  Per workgroup:
// evictable blocks per queue go to a plain store, and blocks with
// (key, id) <= bound to the workgroup's own candidate region (one LDS atomic
// per wave and queue); only a region overflow uses the shared spill list.
#define SCAN_BATCH 256  // blocks per wave per batch: 4 per lane
#define SCAN_WAVES (SCAN_THREADS / SAE_WAVE)

// Four consecutive blocks of one lane, as loaded from HBM.
struct Quad {
    int4 la;
    uint4 off;
    uint32_t m01, m23;
};

__device__ __forceinline__ Quad load_quad(const DevCtx &c, long long base, long long e0, long long N, bool vec)
{
    Quad r;
    r.la = make_int4(0, 0, 0, 0);
    r.off = make_uint4(0, 0, 0, 0);
    r.m01 = r.m23 = 0;
    if (vec && e0 + 3 < N) {
        r.la = *reinterpret_cast<const int4 *>(c.la + base + e0);
        const uint2 m4 = *reinterpret_cast<const uint2 *>(c.meta + base + e0);
        r.off = *reinterpret_cast<const uint4 *>(c.off + base + e0);
        r.m01 = m4.x;
        r.m23 = m4.y;
    } else {
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
        r.la = make_int4(l[0], l[1], l[2], l[3]);
        r.off = make_uint4(o[0], o[1], o[2], o[3]);
        r.m01 = m[0] | (m[1] << 16);
        r.m23 = m[2] | (m[3] << 16);
    }
    return r;
}

__global__ void __launch_bounds__(SCAN_THREADS) k_scan(DevCtx c, SelectArgs a)
{
    __shared__ ScoreTab tab;
    __shared__ unsigned long long thr_s[SAE_MAX_QUEUES];
    __shared__ uint32_t nev_s[SAE_MAX_QUEUES];
    __shared__ uint32_t cnt_s[SAE_MAX_QUEUES];
    __shared__ uint32_t st_s;
    __shared__ int32_t s_la[SCAN_WAVES][SCAN_BATCH];
    __shared__ uint32_t s_off[SCAN_WAVES][SCAN_BATCH];
    __shared__ uint16_t s_meta[SCAN_WAVES][SCAN_BATCH];
    __shared__ uint16_t s_list[SCAN_WAVES][3][SCAN_BATCH];
    const int inst = blockIdx.y;
    const int wg = blockIdx.x;
    const int Q = c.Q;
    const long long N = c.N;
    const long long base = (long long)inst * N;
    const int lane = lane_id();
    const int wave = threadIdx.x / SAE_WAVE;
    load_score_tab(tab, c.state[inst], c);
    if (threadIdx.x < SAE_MAX_QUEUES) {
        thr_s[threadIdx.x] = (threadIdx.x < Q) ? c.thr[(long long)inst * Q + threadIdx.x] : 0ull;
        nev_s[threadIdx.x] = 0;
        cnt_s[threadIdx.x] = 0;
    }
    if (threadIdx.x == 0) st_s = 0;
    __syncthreads();

    // queue kind of every queue, 2 bits each
    uint32_t kinds = 0;
    for (int q = 0; q < SAE_MAX_QUEUES; ++q) kinds |= ((uint32_t)tab.kind[q] & 3u) << (2 * q);

    const int now = a.now;
    unsigned long long cnt_lo = 0, cnt_hi = 0;  // 16-bit evictable counters, queues 0-3 / 4-7
    uint32_t st = 0;
    const bool vec = ((N & 3) == 0);
    const long long nb = (N + SCAN_BATCH - 1) / SCAN_BATCH;
    const long long gw = (long long)wg * SCAN_WAVES + wave;
    const long long tw = (long long)gridDim.x * SCAN_WAVES;
    const long long rbase = ((long long)inst * c.scan_gx + wg) * Q;
    unsigned long long *reg = c.creg + rbase * SAE_CAND_REGION;
    unsigned long long *spill = c.spill + (long long)inst * Q * c.cand_cap;
    uint32_t *spill_n = c.spill_n + (long long)inst * Q;
    int32_t *wla = s_la[wave];
    uint32_t *woff = s_off[wave];
    uint16_t *wmeta = s_meta[wave];

    // append (key, id) of an evictable block if it is within its queue's bound
    auto emit = [&](bool act, int q, uint32_t key, long long b) {
        const unsigned long long comp = ((unsigned long long)key << 32) | (uint32_t)b;
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
            if (in_e && pos < SAE_CAND_REGION) reg[(long long)qq * SAE_CAND_REGION + pos] = comp;
            // beyond the region: one atomic per wave on the queue's spill list
            const unsigned long long ms = __ballot(in_e && pos >= SAE_CAND_REGION);
            if (ms) {
                const int ls = __ffsll((long long)ms) - 1;
                uint32_t sb = 0;
                if (lane == ls) sb = atomicAdd(&spill_n[qq], (uint32_t)__popcll(ms));
                sb = __shfl(sb, ls, SAE_WAVE);
                if (in_e && pos >= SAE_CAND_REGION) {
                    const uint32_t sp = sb + (uint32_t)__popcll(ms & lanemask_lt());
                    if (sp < (uint32_t)c.cand_cap) spill[(long long)qq * c.cand_cap + sp] = comp;
                }
            }
            em &= ~mq;
        }
    };

    // software pipeline: the next batch's loads are in flight while this one is scored
    Quad nxt = {};
    if (gw < nb) nxt = load_quad(c, base, gw * SCAN_BATCH + lane * 4, N, vec);
    for (long long bi = gw; bi < nb; bi += tw) {  // wave-uniform
        const long long b0 = bi * SCAN_BATCH;
        const Quad cur = nxt;
        *reinterpret_cast<int4 *>(wla + lane * 4) = cur.la;
        *reinterpret_cast<uint4 *>(woff + lane * 4) = cur.off;
        *reinterpret_cast<uint2 *>(wmeta + lane * 4) = make_uint2(cur.m01, cur.m23);
        if (bi + tw < nb) nxt = load_quad(c, base, (bi + tw) * SCAN_BATCH + lane * 4, N, vec);
        // kind lists (block indices within the batch)
        uint32_t n0 = 0, n1 = 0, n2 = 0;
        const uint32_t mreg[4] = {cur.m01 & 0xFFFFu, cur.m01 >> 16, cur.m23 & 0xFFFFu, cur.m23 >> 16};
        const unsigned long long lt = lanemask_lt();
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t m = mreg[j];
            const int idx = lane * 4 + j;
            const int q = meta_queue(m);
            const bool ev = meta_evictable(m) && q < Q;
            const int kind = (int)((kinds >> (2 * q)) & 3u);
            const int cls = !ev ? 3 : (kind == SAE_KIND_LOGNORMAL ? 0 : (kind == SAE_KIND_STRUCTURAL ? 1 : 2));
            if (ev) {
                const unsigned long long inc = 1ull << (16 * (q & 3));
                if (q < 4) cnt_lo += inc;
                else cnt_hi += inc;
            }
            const unsigned long long b0m = __ballot(cls == 0);
            const unsigned long long b1m = __ballot(cls == 1);
            const unsigned long long b2m = __ballot(cls == 2);
            if (cls == 0) s_list[wave][0][n0 + __popcll(b0m & lt)] = (uint16_t)idx;
            if (cls == 1) s_list[wave][1][n1 + __popcll(b1m & lt)] = (uint16_t)idx;
            if (cls == 2) s_list[wave][2][n2 + __popcll(b2m & lt)] = (uint16_t)idx;
            n0 += (uint32_t)__popcll(b0m);
            n1 += (uint32_t)__popcll(b1m);
            n2 += (uint32_t)__popcll(b2m);
        }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        __builtin_amdgcn_wave_barrier();
        // log-normal queues
        for (uint32_t i0 = 0; i0 < n0; i0 += SAE_WAVE) {
            const bool act = i0 + lane < n0;
            const int idx = act ? s_list[wave][0][i0 + lane] : 0;
            const uint32_t m = wmeta[idx];
            const uint32_t key = key_lognormal(now, wla[idx], m, tab, st);
            emit(act, meta_queue(m), key, b0 + idx);
        }
        // structural queues
        for (uint32_t i0 = 0; i0 < n1; i0 += SAE_WAVE) {
            const bool act = i0 + lane < n1;
            const int idx = act ? s_list[wave][1][i0 + lane] : 0;
            const uint32_t m = wmeta[idx];
            const uint32_t key = key_structural(now, wla[idx], m, woff[idx], tab, st);
            emit(act, meta_queue(m), key, b0 + idx);
        }
        // evict-first and recency queues
        for (uint32_t i0 = 0; i0 < n2; i0 += SAE_WAVE) {
            const bool act = i0 + lane < n2;
            const int idx = act ? s_list[wave][2][i0 + lane] : 0;
            const uint32_t m = wmeta[idx];
            const int kind = (int)((kinds >> (2 * meta_queue(m))) & 3u);
            const uint32_t key = key_cheap(kind, now, wla[idx], m, tab, st);
            emit(act, meta_queue(m), key, b0 + idx);
        }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        __builtin_amdgcn_wave_barrier();
    }
    for (int q = 0; q < Q; ++q) {
        const uint32_t v = (uint32_t)(((q < 4 ? cnt_lo : cnt_hi) >> (16 * (q & 3))) & 0xFFFFull);
        if (v) atomicAdd(&nev_s[q], v);
    }
    if (st) atomicOr(&st_s, st);
    __syncthreads();
    if (threadIdx.x < Q) {
        c.nev_part[rbase + threadIdx.x] = nev_s[threadIdx.x];
        c.creg_n[rbase + threadIdx.x] = min(cnt_s[threadIdx.x], (uint32_t)SAE_CAND_REGION);
    }
    if (threadIdx.x == 0) set_status(c.status, st_s);
}

// Pool-scan engine, step 4: exact k smallest (key, id) of one (instance,
// queue).  The candidates (every evictable block of the queue with
// (key, id) <= bound) are gathered into LDS; if the bound admitted fewer than
// needed, or more than fit, the workgroup instead streams the instance's pool
// and radix-selects exactly (slow; SAE_ST_SELECT_FALLBACK).
__global__ void __launch_bounds__(SEL_THREADS) k_select(DevCtx c, SelectArgs a, int P)
{
    extern __shared__ unsigned long long el[];  // [LCAP]
    __shared__ BoundScratch bs;
    __shared__ SelState st;
    __shared__ ScoreTab tab;
    __shared__ uint32_t offs[2048 + 1];
    __shared__ uint32_t nev_s, lcount, wsum[16];
    const int q = blockIdx.x;
    const int inst = blockIdx.y;
    const int Q = c.Q;
    const int gx = c.scan_gx;
    const long long iq = (long long)inst * Q + q;
    const long long N = c.N;
    const long long base = (long long)inst * N;
    const int tid = threadIdx.x;
    if (tid == 0) {
        nev_s = 0;
        lcount = 0;
    }
    load_score_tab(tab, c.state[inst], c);
    __syncthreads();
    // evictable count and candidate-region offsets (exclusive scan over workgroups)
    uint32_t nv = 0, r0 = 0, r1 = 0;
    const int w0 = 2 * tid, w1 = 2 * tid + 1;
    if (w0 < gx) {
        nv += c.nev_part[((long long)inst * gx + w0) * Q + q];
        r0 = c.creg_n[((long long)inst * gx + w0) * Q + q];
    }
    if (w1 < gx) {
        nv += c.nev_part[((long long)inst * gx + w1) * Q + q];
        r1 = c.creg_n[((long long)inst * gx + w1) * Q + q];
    }
    {
        uint32_t v = wave_incl_scan(nv);
        if (lane_id() == 63 && v) atomicAdd(&nev_s, v);
        uint32_t loc = r0 + r1;
        uint32_t inc = wave_incl_scan(loc);
        if (lane_id() == 63) wsum[tid >> 6] = inc;
        __syncthreads();
        uint32_t pre = 0;
        for (int w = 0; w < (tid >> 6); ++w) pre += wsum[w];
        const uint32_t ex = pre + inc - loc;
        if (w0 < gx) offs[w0] = ex;
        if (w1 < gx) offs[w1] = ex + r0;
        if (tid == 0) {
            uint32_t t = 0;
            for (int w = 0; w < 16; ++w) t += wsum[w];
            offs[2048] = t;
        }
    }
    __syncthreads();
    const uint32_t nev = nev_s;
    const uint32_t total_r = offs[2048];
    const uint32_t ns = c.spill_n[iq];
    const uint32_t nsp = ns < (uint32_t)c.cand_cap ? ns : (uint32_t)c.cand_cap;
    const uint32_t nc = total_r + nsp;
    const uint32_t need = (uint32_t)min((long long)inst_k(a, inst, c.max_k), (long long)nev);
    const bool fb = (a.flags & SAE_SS_FORCE_FALLBACK) || ns > (uint32_t)c.cand_cap || nc < need || nc > LCAP;
    if (tid == 0) {
        if (fb && need > 0) set_status(c.status, SAE_ST_SELECT_FALLBACK);
        uint32_t *dbg = c.sel_stats + iq * 4;
        dbg[0] = nev;
        dbg[1] = total_r;
        dbg[2] = ns;
        dbg[3] = fb ? 1u : 0u;
    }
    uint32_t dummy = 0;

    if (!fb) {
        // gather the candidates: index math first, then every load in flight
        const unsigned long long *reg = c.creg + ((long long)inst * gx) * Q * SAE_CAND_REGION;
        {
            unsigned long long ev[LCAP / SEL_THREADS];
#pragma unroll
            for (int m = 0; m < LCAP / SEL_THREADS; ++m) {
                const uint32_t i = tid + (uint32_t)m * SEL_THREADS;
                ev[m] = 0;
                if (i < total_r) {
                    int lo = 0, hi = gx - 1;  // last region with offs <= i
                    while (lo < hi) {
                        const int mid = (lo + hi + 1) >> 1;
                        if (offs[mid] <= i) lo = mid;
                        else hi = mid - 1;
                    }
                    ev[m] = reg[((long long)lo * Q + q) * SAE_CAND_REGION + (i - offs[lo])];
                }
            }
#pragma unroll
            for (int m = 0; m < LCAP / SEL_THREADS; ++m) {
                const uint32_t i = tid + (uint32_t)m * SEL_THREADS;
                if (i < total_r) el[i] = ev[m];
            }
        }
        const unsigned long long *spill = c.spill + iq * c.cand_cap;
        for (uint32_t j = tid; j < nsp; j += blockDim.x) el[total_r + j] = spill[j];
        __syncthreads();
        if (need > 0 && need < nc) {
            const unsigned long long T = lds_select_bound(el, (int)nc, need, bs);
            // keep the `need` elements <= T, packed at the front
            unsigned long long mine[LCAP / SEL_THREADS];
#pragma unroll
            for (int j = 0; j < LCAP / SEL_THREADS; ++j) {
                const int i = tid + j * SEL_THREADS;
                mine[j] = (i < (int)nc) ? el[i] : ~0ull;
            }
            __syncthreads();
#pragma unroll
            for (int j = 0; j < LCAP / SEL_THREADS; ++j) {
                if (mine[j] <= T) {
                    const uint32_t pos = atomicAdd(&lcount, 1u);
                    el[pos] = mine[j];
                }
            }
        }
        __syncthreads();
    } else {
        // exact slow path: stream the pool for this queue
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
            for (int i = tid; i < SAE_BINS; i += blockDim.x) bs.hist[i] = 0;
            __syncthreads();
            const unsigned long long pre = st.prefix[0];
            for_each([&](unsigned long long e) {
                if (p == 0 || (e >> (s + w)) == pre) atomicAdd(&bs.hist[(uint32_t)(e >> s) & ((1u << w) - 1u)], 1u);
            });
            __syncthreads();
            find_crossing(bs.hist, 1, st.rem, st.active, st.cr, st.seg_tot);
            sel_step(st, 1, s, w, p == 5);
        }
        for_each([&](unsigned long long e) {
            if (sel_take(st, 0, e)) {
                const uint32_t pos = atomicAdd(&lcount, 1u);
                if (pos < (uint32_t)P) el[pos] = e;
            }
        });
        __syncthreads();
    }
    // sort the selection and write it out
    const uint32_t out = min(need, (uint32_t)P);
    const int PS = P < 256 ? 256 : P;
    for (int i = tid + (int)out; i < PS; i += blockDim.x) el[i] = ~0ull;
    __syncthreads();
    sort_lds(el, PS);
    const long long ob = iq * c.max_k;
    for (uint32_t j = tid; j < out; j += blockDim.x) {
        const unsigned long long e = el[j];
        a.victims[ob + j] = (int32_t)(uint32_t)(e & 0xFFFFFFFFull);
        if (a.scores) a.scores[ob + j] = __uint_as_float((uint32_t)(e >> 32));
        c.sel[ob + j] = e;
    }
    if (tid == 0) {
        a.count[iq] = (int32_t)out;
        c.sel_count[iq] = (int32_t)out;
        c.spill_n[iq] = 0;
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
    hipError_t e;
    // step 1: sample
    const size_t lds_sample = (size_t)c.Q * SAE_SBINS * sizeof(uint32_t);
    hipLaunchKernelGGL(k_sample, dim3(SAMPLE_WGS, c.n_inst), dim3(SCAN_THREADS), lds_sample, s, c, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // step 2: candidate bounds
    const size_t lds_el = (size_t)LCAP * sizeof(unsigned long long);
    if ((e = allow_lds((const void *)k_threshold, lds_el)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_threshold, dim3(c.Q, c.n_inst), dim3(SEL_THREADS), lds_el, s, c, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // step 3: streaming pass
    if (ev0 && (e = hipEventRecord(ev0, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_scan, dim3(c.scan_gx, c.n_inst), dim3(SCAN_THREADS), 0, s, c, a);
    e = hipGetLastError();
    if (e == hipSuccess && ev1) e = hipEventRecord(ev1, s);
    if (e != hipSuccess) return e;
    // step 4: per (queue, instance) exact select
    const int P = pow2_at_least(c.max_k);
    if ((e = allow_lds((const void *)k_select, lds_el)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_select, dim3(c.Q, c.n_inst), dim3(SEL_THREADS), lds_el, s, c, a, P);
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
