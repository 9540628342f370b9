// Eviction-feedback learners: Algorithms 2, 3 and 4 and the decay-power
// learner, one workgroup per instance.  fp32 in the order the
// algorithms state them (built with -ffp-contract=off, so no operation is
// fused); Algorithm 4's moments are exact integer sums rounded once.
#include "sae_internal.h"

namespace {

__device__ __forceinline__ float clampf(float x, float lo, float hi) { return fminf(fmaxf(x, lo), hi); }

// floor(0.99 x) in integers: the decay factor lambda = 0.99 of the eviction
// feedback counters, applied without rounding error.
__device__ __forceinline__ int32_t decay99(int32_t x) { return (int32_t)(((long long)x * 99) / 100); }

// 128-bit unsigned sum kept as two 64-bit halves.
struct U128 {
    unsigned long long lo, hi;
};
__device__ __forceinline__ U128 add128(U128 a, U128 b)
{
    U128 r;
    r.lo = a.lo + b.lo;
    r.hi = a.hi + b.hi + (r.lo < a.lo ? 1ull : 0ull);
    return r;
}

// Algorithm 4 for every log-normal queue with more than 20 buffered
// intervals.  The workgroup's threads split the buffers; X = ln(dt) * 2^24
// is an exact integer (ivl_scaled_ln), so the sums S1 = sum X, S2 = sum X^2
// are exact in any order.  Thread q then rounds:
// m = S1 / n * 2^-24, v = max(S2 / n * 2^-48 - m m, 0) in double,
// mu_s = fl32(m), sigma_s = fl32(sqrt v), followed by the fp32 EMA.
constexpr int kLearnThreads = 1024;

// Position of the k-th set bit of m (k < popcount(m)).
__device__ __forceinline__ int nth_bit(uint32_t m, int k)
{
    for (int j = 0; j < k; ++j) m &= m - 1u;
    return __ffs(m) - 1;
}

// Per-wave partial sums of Algorithm 4, kept in LDS between its two halves.
struct Alg4Sums {
    long long s1[kLearnThreads / SAE_WAVE];
    unsigned long long s2lo[kLearnThreads / SAE_WAVE], s2hi[kLearnThreads / SAE_WAVE];
};

__device__ __forceinline__ long long ivl_lo(const InstState &s, int q)
{
    const long long n = s.ivl_n[q];
    return s.ivl_start[q] > n - SAE_IVL_CAP ? s.ivl_start[q] : n - SAE_IVL_CAP;
}

// First half, on all threads: the log-normal queues with more than 20
// buffered intervals (returned as a bit mask, the same on every thread) and
// the exact sums of their buffers, one queue per wave group; ends with a
// workgroup barrier when the mask is not empty.
__device__ uint32_t alg4_sums(const DevCtx &c, int inst, const InstState &s, int t, Alg4Sums &w)
{
    constexpr int NW = kLearnThreads / SAE_WAVE;
    constexpr int BATCH = 8;  // loads a thread has in flight together
    const int lane = t % SAE_WAVE, wave = t / SAE_WAVE;
    uint32_t due = 0;
    for (int q = 0; q < c.Q; ++q)
        if (((c.ln_mask >> q) & 1u) && s.ivl_n[q] - ivl_lo(s, q) > 20) due |= 1u << q;
    if (!due) return 0;
    // wave v sums part of the (v mod nd)-th due queue's buffer
    const int nd = __popc(due);
    const int qi = wave % nd;
    const int q = nth_bit(due, qi);
    const int wq = wave / nd, nwq = (NW - 1 - qi) / nd + 1;
    const long long n = s.ivl_n[q];
    const long long lo = ivl_lo(s, q);
    const int32_t *ring = c.ivl + ((long long)inst * c.Q + q) * SAE_IVL_CAP;
    const long long stride = (long long)nwq * SAE_WAVE;
    long long s1 = 0;
    U128 s2 = {0ull, 0ull};
    for (long long b0 = lo + (long long)wq * SAE_WAVE; b0 < n; b0 += BATCH * stride) {
        int32_t d[BATCH];
#pragma unroll
        for (int k = 0; k < BATCH; ++k) {  // unconditional loads at clamped positions
            const long long p = b0 + lane + k * stride;
            d[k] = ring[(p < n ? p : lo) & (SAE_IVL_CAP - 1)];
        }
#pragma unroll
        for (int k = 0; k < BATCH; ++k) {
            const long long p = b0 + lane + k * stride;
            const long long X = p < n ? ivl_scaled_ln(d[k]) : 0;
            const unsigned long long X2 = (unsigned long long)X * (unsigned long long)X;
            s1 += X;
            s2 = add128(s2, U128{X2, 0ull});
        }
    }
    for (int o = SAE_WAVE / 2; o > 0; o >>= 1) {
        s1 += __shfl_xor(s1, o);
        U128 u;
        u.lo = __shfl_xor(s2.lo, o);
        u.hi = __shfl_xor(s2.hi, o);
        s2 = add128(s2, u);
    }
    if (lane == 0) {
        w.s1[wave] = s1;
        w.s2lo[wave] = s2.lo;
        w.s2hi[wave] = s2.hi;
    }
    __syncthreads();
    return due;
}

// Second half, thread j < popcount(due): the j-th due queue's moments and EMA.
__device__ void alg4_finish(InstState &s, int j, uint32_t due, const Alg4Sums &w)
{
    constexpr int NW = kLearnThreads / SAE_WAVE;
    const int nd = __popc(due);
    const int q = nth_bit(due, j);
    long long S1 = 0;
    U128 S2 = {0ull, 0ull};
    for (int v = j; v < NW; v += nd) {
        S1 += w.s1[v];
        S2 = add128(S2, U128{w.s2lo[v], w.s2hi[v]});
    }
    const long long n = s.ivl_n[q];
    const long long lo = ivl_lo(s, q);
    const double cnt = (double)(n - lo);
    const double m = ((double)S1 / cnt) * 0x1p-24;
    const double s2d = (double)S2.hi * 0x1p64 + (double)S2.lo;
    double v = (s2d / cnt) * 0x1p-48 - m * m;
    if (v < 0.0) v = 0.0;
    const float mu_s = (float)m;
    const float sd_s = (float)sqrt(v);
    s.mu[q] = s.mu[q] + s.beta_ln * (mu_s - s.mu[q]);
    const float sg = s.sigma[q] + s.beta_ln * (sd_s - s.sigma[q]);
    s.sigma[q] = fmaxf(sg, 0.1f);
    s.ivl_start[q] = lo > n - 200 ? lo : n - 200;  // keep the last 200
}

// Decay-power learner (App. B) over the positional bins: hit rate per bin,
// front (bins 0-3) and back (bins 4-7) averages over bins with events,
// estimate 1 / (back / front + 0.1), EMA by beta and clip to [0.3, 3.0].
__device__ void decay_power(InstState &s)
{
    int32_t ev[SAE_N_BINS];
    int32_t total = 0;
    for (int b = 0; b < SAE_N_BINS; ++b) {
        ev[b] = s.bin_hits[b] + s.bin_missed[b];
        total += ev[b];
    }
    if (total <= 20) return;
    float fsum = 0.0f, bsum = 0.0f;
    int fn = 0, bn = 0;
    for (int b = 0; b < SAE_N_BINS; ++b) {
        if (ev[b] == 0) continue;
        const float rate = (float)s.bin_hits[b] / (float)ev[b];
        if (b < SAE_N_BINS / 2) {
            fsum = fsum + rate;
            ++fn;
        } else {
            bsum = bsum + rate;
            ++bn;
        }
    }
    if (fn == 0 || bn == 0) return;
    const float front = fsum / (float)fn;
    const float back = bsum / (float)bn;
    if (!(front > 0.0f)) return;
    const float ratio = back / front;
    const float est = 1.0f / (ratio + 0.1f);
    s.gamma = clampf(s.gamma + s.beta * (est - s.gamma), 0.3f, 3.0f);
    for (int b = 0; b < SAE_N_BINS; ++b) s.bin_hits[b] = s.bin_missed[b] = 0;
}

// The appendix text's token-weight rule for type t (one lane): an EMA toward
// 1 + 5 r_miss + 2 r_reuse, counters decayed by floor(0.99 x).
__device__ void token_weight_ema(InstState &s, int t)
{
    const int32_t ev = s.evicted[t], mi = s.missed[t], h = s.type_hits[t], a = s.type_added[t];
    const float r_miss = ev > 0 ? (float)mi / (float)ev : 0.0f;
    const float r_reuse = (h + a) > 0 ? (float)h / (float)(h + a) : 0.0f;
    const float target = 1.0f + r_miss * 5.0f + r_reuse * 2.0f;
    s.w[t] = clampf((1.0f - s.eta) * s.w[t] + s.eta * target, 0.1f, 5.0f);
    s.evicted[t] = decay99(ev);
    s.missed[t] = decay99(mi);
    s.type_hits[t] = decay99(h);
    s.type_added[t] = decay99(a);
}

// The appendix text's queue-weight rule over all queues (one lane):
// relative efficiency (hits per share of the cached blocks) to the power 1/T,
// blended as beta alpha + (1 - beta) target.
__device__ void queue_weights_rel(const DevCtx &c, InstState &s)
{
    int32_t total = 0;
    for (int q = 0; q < c.Q; ++q) total += s.resident[q];
    float E[SAE_MAX_QUEUES];
    float e_sum = 0.0f;
    int m = 0;
#pragma unroll
    for (int q = 0; q < SAE_MAX_QUEUES; ++q) {
        E[q] = 0.0f;
        if (q < c.Q && c.kind[q] != SAE_KIND_EVICT_FIRST && s.resident[q] > 0 && total > 0) {
            const float share = (float)s.resident[q] / (float)total;
            E[q] = (float)s.hits[q] / share;
            e_sum = e_sum + E[q];
            ++m;
        }
    }
    if (m > 0) {
        const float e_mean = e_sum / (float)m;
        if (e_mean > 0.0f) {
#pragma unroll
            for (int q = 0; q < SAE_MAX_QUEUES; ++q) {
                if (!(q < c.Q && c.kind[q] != SAE_KIND_EVICT_FIRST && s.resident[q] > 0)) continue;
                const float x = E[q] / e_mean;
                const float tgt = (s.T == 1.0f || x == 0.0f) ? x : dsr::exp(dsr::ln(x) / s.T);
                s.alpha[q] = clampf(s.beta * s.alpha[q] + (1.0f - s.beta) * tgt, 0.1f, 3.0f);
            }
        }
    }
    for (int q = 0; q < c.Q; ++q) {
        if (c.kind[q] == SAE_KIND_EVICT_FIRST) continue;
        s.hits[q] = 0;
        s.evictions[q] = 0;
    }
}

// Token weight of type t (Algorithm 3).  A type whose evicted blocks keep
// being asked for again is being evicted too eagerly: once more than ten of
// its blocks have gone, its weight is multiplied by 1 + eta * (returns per
// eviction) and kept in [0.1, 5].  Both counts then shrink by lambda, whether
// or not the weight moved.  The fp32 operations run in this order: ratio,
// times eta, plus one, times the weight.
__device__ __forceinline__ void token_weight_alg3(InstState &s, int t)
{
    const int32_t ev = s.evicted[t], mi = s.missed[t];
    if (ev > 10) s.w[t] = clampf(s.w[t] * (1.0f + s.eta * ((float)mi / (float)ev)), 0.1f, 5.0f);
    s.evicted[t] = decay99(ev);
    s.missed[t] = decay99(mi);
}

// Queue weight of queue q (Algorithm 2).  The target is 1 plus the queue's
// prefix-match hits per eviction, scaled by 1 / T; with more than five
// evictions since the last run, alpha moves the fraction beta of its distance
// to the target and is kept in [0.1, 3].  The queue's counts restart in any
// case.  fp32 order: ratio, over T, plus one, minus alpha, times beta, plus
// alpha.
__device__ __forceinline__ void queue_weight_alg2(InstState &s, int q)
{
    const int32_t h = s.hits[q], e = s.evictions[q];
    if (e > 5) {
        const float target = 1.0f + ((float)h / (float)e) / s.T;
        s.alpha[q] = clampf(s.alpha[q] + s.beta * (target - s.alpha[q]), 0.1f, 3.0f);
    }
    s.hits[q] = 0;
    s.evictions[q] = 0;
}

// Token-weight, queue-weight and decay-power learners on the lanes of one
// wave, which touch disjoint fields: lane l < 5 updates token type l
// (Algorithm 3 or the text's rule), lane 8 + q queue q (Algorithm 2), lane 16
// every queue (the text's rule), lane 63 gamma.
__device__ void learners_23_gamma(const DevCtx &c, InstState &s, int l)
{
    if (l < SAE_N_TYPES) {
        if (s.learn & SAE_LEARN_TOKEN_EMA) {
            token_weight_ema(s, l);
        } else if (s.learn & SAE_LEARN_TOKEN_WEIGHTS) {
            token_weight_alg3(s, l);
        }
    } else if (l == 16) {
        if (s.learn & SAE_LEARN_QUEUE_REL) queue_weights_rel(c, s);
    } else if (l >= 8 && l < 8 + c.Q) {
        const int q = l - 8;
        if ((s.learn & SAE_LEARN_QUEUE_WEIGHTS) && c.kind[q] != SAE_KIND_EVICT_FIRST) queue_weight_alg2(s, q);
    } else if (l == SAE_WAVE - 1) {
        if (s.learn & SAE_LEARN_DECAY_POWER) decay_power(s);
    }
}

// One workgroup of 1024 threads per instance.  The instance state is copied
// into LDS while the striped counter copies are read (one memory round trip)
// and summed per field in LDS; thread f folds field f into the copy.  Then, if
// asked and due, Algorithm 4 sums on all threads and then finishes on wave 0
// while wave 1 runs the other learners on the copy, which is written back at
// the end.
static_assert(sizeof(InstState) % 4 == 0, "InstState is copied as 32-bit words");
__global__ void __launch_bounds__(kLearnThreads) k_feedback(DevCtx c, uint32_t flags, int learn)
{
    constexpr int NWORDS = (int)(sizeof(InstState) / 4);
    __shared__ InstState s;
    __shared__ int due;
    const int inst = blockIdx.x;
    const int f = threadIdx.x;
    __shared__ int32_t fsum[SAE_CF_STRIDE];
    uint32_t *gw = reinterpret_cast<uint32_t *>(c.state + inst);
    uint32_t *lw = reinterpret_cast<uint32_t *>(&s);
    for (int w = f; w < NWORDS; w += kLearnThreads) lw[w] = gw[w];
    if (f < SAE_CF_STRIDE) fsum[f] = 0;
    // every (copy, field) word of the striped counters: all loads in flight together
    constexpr int NC = SAE_CSLOTS * SAE_CF_STRIDE / kLearnThreads;
    static_assert(NC * kLearnThreads == SAE_CSLOTS * SAE_CF_STRIDE, "counter words split evenly");
    int32_t *cbase = c.cpart + (long long)inst * SAE_CSLOTS * SAE_CF_STRIDE;
    int32_t cv[NC];
#pragma unroll
    for (int j = 0; j < NC; ++j) cv[j] = cbase[f + j * kLearnThreads];
    __syncthreads();
#pragma unroll
    for (int j = 0; j < NC; ++j)
        if (cv[j]) {
            const int e = f + j * kLearnThreads;
            cbase[e] = 0;
            atomicAdd(&fsum[e % SAE_CF_STRIDE], cv[j]);
        }
    __syncthreads();
    const int32_t sum = f < SAE_CF_N ? fsum[f] : 0;
    if (f < SAE_CF_N && sum) {
        if (f < SAE_CF_MISSED) s.evicted[f - SAE_CF_EVICTED] += sum;
        else if (f < SAE_CF_HITS) s.missed[f - SAE_CF_MISSED] += sum;
        else if (f < SAE_CF_EVICTIONS) s.hits[f - SAE_CF_HITS] += sum;
        else if (f < SAE_CF_BHITS) s.evictions[f - SAE_CF_EVICTIONS] += sum;
        else if (f < SAE_CF_BMISS) s.bin_hits[f - SAE_CF_BHITS] += sum;
        else if (f < SAE_CF_THITS) s.bin_missed[f - SAE_CF_BMISS] += sum;
        else if (f < SAE_CF_TADD) s.type_hits[f - SAE_CF_THITS] += sum;
        else if (f < SAE_CF_RES) s.type_added[f - SAE_CF_TADD] += sum;
        else s.resident[f - SAE_CF_RES] += sum;
    }
    if (f == 0) due = learn && (s.pending || (flags & SAE_FB_FORCE));
    __syncthreads();
    if (due) {
        __shared__ Alg4Sums a4;
        const uint32_t ln_due = ((s.learn & SAE_LEARN_LOGNORMAL) && c.ln_mask) ? alg4_sums(c, inst, s, f, a4) : 0u;
        if (f < __popc(ln_due)) alg4_finish(s, f, ln_due, a4);                 // wave 0
        else if (f >= SAE_WAVE && f < 2 * SAE_WAVE) learners_23_gamma(c, s, f - SAE_WAVE);  // wave 1
        __syncthreads();
        if (f == 0) {
            s.pending = 0;
            s.n_updates += 1;
        }
    }
    __syncthreads();
    for (int w = f; w < NWORDS; w += kLearnThreads) gw[w] = lw[w];
}

}  // namespace

hipError_t launch_feedback(const DevCtx &c, uint32_t flags, int learn, hipStream_t s)
{
    hipLaunchKernelGGL(k_feedback, dim3(c.n_inst), dim3(kLearnThreads), 0, s, c, flags, learn);
    return hipGetLastError();
}
