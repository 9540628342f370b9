// Eviction-feedback learners (Algorithms 2 and 3), one thread per instance.
// fp32 throughout, in the order the algorithms state them (built with
// -ffp-contract=off, so no operation is fused).
#include "sae_internal.h"

namespace {

__device__ __forceinline__ float clampf(float x, float lo, float hi) { return fminf(fmaxf(x, lo), hi); }

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
            else s.evictions[f - SAE_CF_EVICTIONS] += sum;
        }
    }
    __syncthreads();
    if (!learn || f != 0) return;
    if (!s.pending && !(flags & SAE_FB_FORCE)) return;
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
    s.pending = 0;
    s.n_updates += 1;
}

}  // namespace

hipError_t launch_feedback(const DevCtx &c, uint32_t flags, int learn, hipStream_t s)
{
    hipLaunchKernelGGL(k_feedback, dim3(c.n_inst), dim3(64), 0, s, c, flags, learn);
    return hipGetLastError();
}
