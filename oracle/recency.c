/*
 * TEST INFRASTRUCTURE — a faster exact CPU selection, the per-queue heap idea
 * of the paper's cost discussion (Sec. 3.2, Algorithm 1), used as a second
 * CPU baseline.  Only tests/ and bench.py's cpu_baseline leg load this
 * library; it shares no code with the HIP path.
 *
 * Per (queue, block type) group of a log-normal or recency queue, P (Eq. 3)
 * depends on dt alone, and the fp32 recipe of dsr.c never lets an older block
 * (larger dt) score more than a factor 1 + 2^-19 above a younger one while P
 * is a normal number (ln rises monotonically, the erfc realisation by at most
 * one ulp over [0, 9]; for a recency queue P = aw / dt is monotone outright).
 * So each group is kept as a list of its evictable blocks in (last_access,
 * id) order, oldest first, and a selection walks the lists from their heads:
 *   1. the first `prefill` blocks of every group (k in use: with P monotone
 *      they already hold the answer) go into a bounded max-heap of k
 *      (bits(P) << 32 | id) keys, whose top B, once k are in, bounds the k-th
 *      smallest key;
 *   2. every list is walked on until a block with P > T' = max(B (1 + 2^-15),
 *      2^-100) (B the heap's current top): every younger block then scores
 *      above T' / (1 + 2^-19) > B, so none of them can enter;
 *   3. the heap's contents, sorted, are the queue's k smallest (P, id).
 * Equal last_access within a group means equal P; the list holds those
 * blocks in id order, and the heap orders them by id anyway.  A structural
 * queue (P also depends on o_b / o_max) is scanned whole into the bounded
 * heap; an evict-first queue (key num_tokens) needs no scoring: its list in
 * (num_tokens, id) order gives the answer directly (done by the caller).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

float oracle_p_lognormal(int32_t dt, float mu, float c);
float oracle_p_structural(int32_t ob, int32_t omax, float gamma);
float oracle_inv_sigma_sqrt2(float sigma);

enum { RL_LOGNORMAL = 2, RL_RECENCY = 3 };

static inline uint32_t rl_f2u(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static inline float rl_u2f(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

/* bounded max-heap of at most k keys */
typedef struct {
    uint64_t *h;
    int32_t n, k;
} rl_heap;

static void rl_sift_down(uint64_t *h, int32_t n, int32_t i)
{
    const uint64_t v = h[i];
    for (;;) {
        int32_t c = 2 * i + 1;
        if (c >= n) break;
        if (c + 1 < n && h[c + 1] > h[c]) ++c;
        if (h[c] <= v) break;
        h[i] = h[c];
        i = c;
    }
    h[i] = v;
}

static void rl_offer(rl_heap *hp, uint64_t key)
{
    uint64_t *h = hp->h;
    if (hp->n < hp->k) {
        int32_t i = hp->n++;
        while (i > 0) {
            const int32_t p = (i - 1) / 2;
            if (h[p] >= key) break;
            h[i] = h[p];
            i = p;
        }
        h[i] = key;
    } else if (hp->k > 0 && key < h[0]) {
        h[0] = key;
        rl_sift_down(h, hp->n, 0);
    }
}

/* sorts the heap's keys ascending in place (heapsort); returns the count */
static int32_t rl_drain(rl_heap *hp, uint32_t *keys, int32_t *ids)
{
    uint64_t *h = hp->h;
    for (int32_t n = hp->n; n > 1; --n) {
        const uint64_t t = h[0];
        h[0] = h[n - 1];
        h[n - 1] = t;
        rl_sift_down(h, n - 1, 0);
    }
    for (int32_t i = 0; i < hp->n; ++i) {
        keys[i] = (uint32_t)(h[i] >> 32);
        ids[i] = (int32_t)(uint32_t)h[i];
    }
    return hp->n;
}

static inline float rl_score(int32_t kind, int32_t now, int32_t la, float aw, float mu, float c)
{
    int32_t dt = now - la;
    if (dt < 0) dt = 0;
    if (dt == 0) return INFINITY;
    const float p = (kind == RL_LOGNORMAL) ? oracle_p_lognormal(dt, mu, c) : 1.0f;
    const float nn = aw * p;
    return nn / (float)dt;
}

/*
 * One log-normal or recency queue: gstart[0..5] delimit the five type groups
 * in gids (each in (last_access, id) order); aw[t] = fl(alpha_q w_t).  Writes
 * the min(k, evictable) smallest (key, id) in order; heap holds k entries.
 * *visited receives the number of blocks scored.  Any prefill >= 0 gives the
 * same result; tests use a small one so that the stopping rule decides.
 */
int32_t oracle_rl_select(int32_t k, int32_t prefill, int32_t now, int32_t kind, float mu, float sigma, const float *aw,
                         const int64_t *gstart, const int32_t *gids, const int32_t *la, uint64_t *heap,
                         uint32_t *out_keys, int32_t *out_ids, int64_t *visited)
{
    rl_heap hp = {heap, 0, k};
    const float c = (kind == RL_LOGNORMAL) ? oracle_inv_sigma_sqrt2(sigma) : 0.0f;
    int64_t pos[5], seen = 0;
    if (k <= 0) {
        *visited = 0;
        return 0;
    }
    for (int t = 0; t < 5; ++t) {
        int64_t i = gstart[t];
        const int64_t end = (gstart[t + 1] - i > prefill) ? i + prefill : gstart[t + 1];
        for (; i < end; ++i) {
            const int32_t b = gids[i];
            const float P = rl_score(kind, now, la[b], aw[t], mu, c);
            rl_offer(&hp, ((uint64_t)rl_f2u(P) << 32) | (uint32_t)b);
        }
        seen += end - gstart[t];
        pos[t] = end;
    }
    for (int t = 0; t < 5; ++t) {
        for (int64_t i = pos[t]; i < gstart[t + 1]; ++i) {
            if (hp.n == k) {
                const float B = rl_u2f((uint32_t)(hp.h[0] >> 32));
                const float T = fmaxf(B * (1.0f + 0x1p-15f), 0x1p-100f);
                const int32_t b = gids[i];
                const float P = rl_score(kind, now, la[b], aw[t], mu, c);
                ++seen;
                if (isfinite(T) && P > T) break;
                rl_offer(&hp, ((uint64_t)rl_f2u(P) << 32) | (uint32_t)b);
            } else {
                const int32_t b = gids[i];
                rl_offer(&hp, ((uint64_t)rl_f2u(rl_score(kind, now, la[b], aw[t], mu, c)) << 32) | (uint32_t)b);
                ++seen;
            }
        }
    }
    *visited = seen;
    return rl_drain(&hp, out_keys, out_ids);
}

/* A structural queue: every evictable block of it (ids[0..n)) into the heap. */
int32_t oracle_struct_select(int32_t k, int32_t now, float gamma, const float *aw, int64_t n, const int32_t *ids,
                             const int32_t *la, const int32_t *tau, const int32_t *ob, const int32_t *omax,
                             uint64_t *heap, uint32_t *out_keys, int32_t *out_ids)
{
    rl_heap hp = {heap, 0, k};
    if (k <= 0) return 0;
    for (int64_t i = 0; i < n; ++i) {
        const int32_t b = ids[i];
        int32_t dt = now - la[b];
        if (dt < 0) dt = 0;
        float P;
        if (dt == 0) {
            P = INFINITY;
        } else {
            const float p = oracle_p_structural(ob[b], omax[b], gamma);
            const float nn = aw[tau[b]] * p;
            P = nn / (float)dt;
        }
        rl_offer(&hp, ((uint64_t)rl_f2u(P) << 32) | (uint32_t)b);
    }
    return rl_drain(&hp, out_keys, out_ids);
}
