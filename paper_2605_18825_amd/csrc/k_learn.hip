// Eviction-feedback learners: Algorithms 2, 3 and 4 and the decay-power
// learner, one workgroup of one wave per instance.  fp32 in the order the
// algorithms state them (built with -ffp-contract=off, so no operation is
// fused); Algorithm 4's moments are exact integer sums rounded once.
#include "sae_internal.h"

namespace {

__device__ __forceinline__ float clampf(float x, float lo, float hi) { return fminf(fmaxf(x, lo), hi); }

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
// intervals.  The wave's 64 lanes split the buffer; x = ln dt in the fp32
// recipe is 0 or >= ln 2, so X = x * 2^24 is an integer and the sums
// S1 = sum X, S2 = sum X^2 are exact in any order.  Lane 0 then rounds:
// m = S1 / n * 2^-24, v = max(S2 / n * 2^-48 - m m, 0) in double,
// mu_s = fl32(m), sigma_s = fl32(sqrt v), followed by the fp32 EMA.
__device__ void lognormal_params(const DevCtx &c, int inst, InstState &s, int lane)
{
    for (int q = 0; q < c.Q; ++q) {
        if (!((c.ln_mask >> q) & 1u)) continue;
        const long long n = s.ivl_n[q];
        const long long lo = s.ivl_start[q] > n - SAE_IVL_CAP ? s.ivl_start[q] : n - SAE_IVL_CAP;
        const long long cnt = n - lo;
        if (cnt <= 20) continue;
        const int32_t *ring = c.ivl + ((long long)inst * c.Q + q) * SAE_IVL_CAP;
        long long s1 = 0;
        U128 s2 = {0ull, 0ull};
        for (long long p = lo + lane; p < n; p += SAE_WAVE) {
            const float x = dsr::ln((float)ring[p % SAE_IVL_CAP]);
            const long long X = (long long)(x * 16777216.0f);
            const unsigned long long X2 = (unsigned long long)X * (unsigned long long)X;
            s1 += X;
            s2 = add128(s2, U128{X2, 0ull});
        }
        for (int o = SAE_WAVE / 2; o > 0; o >>= 1) {
            s1 += __shfl_xor(s1, o);
            U128 t;
            t.lo = __shfl_xor(s2.lo, o);
            t.hi = __shfl_xor(s2.hi, o);
            s2 = add128(s2, t);
        }
        if (lane == 0) {
            const double nd = (double)cnt;
            const double m = ((double)s1 / nd) * 0x1p-24;
            const double s2d = (double)s2.hi * 0x1p64 + (double)s2.lo;
            double v = (s2d / nd) * 0x1p-48 - m * m;
            if (v < 0.0) v = 0.0;
            const float mu_s = (float)m;
            const float sd_s = (float)sqrt(v);
            s.mu[q] = s.mu[q] + s.beta_ln * (mu_s - s.mu[q]);
            const float sg = s.sigma[q] + s.beta_ln * (sd_s - s.sigma[q]);
            s.sigma[q] = fmaxf(sg, 0.1f);
            s.ivl_start[q] = lo > n - 200 ? lo : n - 200;  // keep the last 200
        }
    }
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

// One workgroup of 64 threads per instance: first fold the striped counter
// copies into the instance state (thread f sums field f over the copies),
// then, if asked and due, thread 0 runs the learners.
__global__ void k_feedback(DevCtx c, uint32_t flags, int learn)
{
    const int inst = blockIdx.x;
    InstState &s = c.state[inst];
    const int f = threadIdx.x;
    if (f < SAE_CF_N) {
        int32_t *base = c.cpart + (long long)inst * SAE_CSLOTS * SAE_CF_STRIDE + f;
        int32_t sum = 0;
        for (int k = 0; k < SAE_CSLOTS; ++k) {
            sum += base[k * SAE_CF_STRIDE];
            base[k * SAE_CF_STRIDE] = 0;
        }
        if (sum) {
            if (f < SAE_CF_MISSED) s.evicted[f - SAE_CF_EVICTED] += sum;
            else if (f < SAE_CF_HITS) s.missed[f - SAE_CF_MISSED] += sum;
            else if (f < SAE_CF_EVICTIONS) s.hits[f - SAE_CF_HITS] += sum;
            else if (f < SAE_CF_BHITS) s.evictions[f - SAE_CF_EVICTIONS] += sum;
            else if (f < SAE_CF_BMISS) s.bin_hits[f - SAE_CF_BHITS] += sum;
            else s.bin_missed[f - SAE_CF_BMISS] += sum;
        }
    }
    __syncthreads();
    if (!learn) return;
    if (!s.pending && !(flags & SAE_FB_FORCE)) return;
    if ((s.learn & SAE_LEARN_LOGNORMAL) && c.ln_mask) lognormal_params(c, inst, s, f);
    if (f != 0) return;
    if (s.learn & SAE_LEARN_TOKEN_WEIGHTS) {
        // Algorithm 3: raise the weight of types evicted too aggressively;
        // both counters decay by lambda = 0.99, applied as floor(99 x / 100).
        for (int t = 0; t < SAE_N_TYPES; ++t) {
            int32_t ev = s.evicted[t], mi = s.missed[t];
            if (ev > 10) {
                float rate = (float)mi / (float)ev;
                float step = s.eta * rate;
                float grow = 1.0f + step;
                s.w[t] = clampf(s.w[t] * grow, 0.1f, 5.0f);
            }
            s.evicted[t] = (int32_t)(((long long)ev * 99) / 100);
            s.missed[t] = (int32_t)(((long long)mi * 99) / 100);
        }
    }
    if (s.learn & SAE_LEARN_QUEUE_WEIGHTS) {
        // Algorithm 2: EMA of the queue weight toward 1 + efficiency / T.
        for (int q = 0; q < c.Q; ++q) {
            if (c.kind[q] == SAE_KIND_EVICT_FIRST) continue;
            int32_t h = s.hits[q], e = s.evictions[q];
            if (e > 5) {
                float eff = (float)h / (float)e;
                float target = 1.0f + eff / s.T;
                float diff = target - s.alpha[q];
                float stepq = s.beta * diff;
                s.alpha[q] = clampf(s.alpha[q] + stepq, 0.1f, 3.0f);
            }
            s.hits[q] = 0;
            s.evictions[q] = 0;
        }
    }
    if (s.learn & SAE_LEARN_DECAY_POWER) decay_power(s);
    s.pending = 0;
    s.n_updates += 1;
}

}  // namespace

hipError_t launch_feedback(const DevCtx &c, uint32_t flags, int learn, hipStream_t s)
{
    hipLaunchKernelGGL(k_feedback, dim3(c.n_inst), dim3(64), 0, s, c, flags, learn);
    return hipGetLastError();
}
