/*
 * TEST INFRASTRUCTURE — CPU oracle, fp32 scoring recipe.
 *
 * Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may
 * load this file's library.  It shares no code with the HIP path.
 *
 * What it computes (paper, Section 3.1):
 *   Eq. 1  p_q(b) = 1 - F_LN(dt; mu_q, sigma_q)       (chat / agent queues)
 *   Eq. 2  p_q(b) = 1 - (o_b / o_max)^gamma            (structural queue)
 *   Eq. 3  P(b)   = alpha_q * w_tau(b) * p_q(b) / dt    (global priority)
 * plus the Algorithm 1 stage-1 key num_tokens(b) for the evict-first queue.
 *
 * The selection that follows (an argmin over P with ties by block id) is
 * decided in fp32, so both the oracle and the kernels realise Eq. 1-3 with
 * the same deterministic fp32 recipe: only IEEE-754 binary32 + - * /,
 * fmaf (single rounding), int<->float conversion and exact bit operations,
 * in a fixed order.  Build with -ffp-contract=off and without fast-math.
 *
 *   ln(x)   : x = 2^e * m, m in (sqrt(1/2), sqrt(2)], ln m = 2 atanh(s),
 *             s = (m-1)/(m+1), atanh by its Taylor series s + s^3/3 + ... + s^9/9
 *             (coefficients 1/(2j+1)); ln 2 split into a 15-bit head and a
 *             tail (Cody & Waite, 1980).
 *   exp(y)  : y = n ln2 + r, n = rint(y / ln 2) (Cody & Waite reduction),
 *             exp(r) by its Taylor series to r^7/7!, scaled by 2^n through
 *             the exponent field.  exp(y) = 0 below y = -86 (keeps every
 *             result a normal number), +inf above 88.
 *   erfc(x) : x >= 0, the Chebyshev-fitted form t*exp(-x^2 + g(t)),
 *             t = 1/(1 + x/2), g a degree-9 polynomial, published by
 *             Press, Teukolsky, Vetterling & Flannery, Numerical Recipes
 *             (2nd ed., Sec. 6.2), fractional error < 1.2e-7.  x^2 is carried
 *             as an exact head+tail pair into the exponential.  erfc(0) = 1
 *             exactly; erfc(x) = 0 for x >= 9.
 *   Eq. 1   : 1 - F_LN(dt) = erfc(u)/2 with u = (ln dt - mu) / (sigma sqrt 2);
 *             for u < 0 it is 1 - erfc(-u)/2 (same value, no cancellation).
 *   Eq. 2   : r = o_b / o_max (o_max = 0 gives r = 0); r^gamma is r itself
 *             for r in {0, 1} or gamma == 1, else exp(gamma ln r).
 *   Eq. 3   : P = ((alpha_q * w_tau) * p) / dt, dt = 0 gives +inf.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

/* ---- constants, each a rounding of an exact mathematical value ---------- */
static const float LN2_HI  = 0x1.62e400p-1f;  /* ln 2 cut to 15 significant bits */
static const float LN2_LO  = 0x1.7f7d1cp-20f; /* fl32(ln 2 - LN2_HI)              */
static const float INV_LN2 = 0x1.715476p+0f;  /* fl32(1 / ln 2)                   */
static const float SQRT2   = 0x1.6a09e6p+0f;  /* fl32(sqrt 2)                     */
static const float RND     = 0x1.8p+23f;      /* 1.5 * 2^23: round-to-integer     */

static inline uint32_t f2u(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static inline float u2f(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

/* 2^n for n in [-126, 127] */
static inline float pow2i(int n) { return u2f((uint32_t)(n + 127) << 23); }

/* exp(r) for |r| <= ~0.35: Taylor series 1 + r + r^2/2! + ... + r^7/7! */
static float exp_taylor(float r)
{
    const float c7 = 1.0f / 5040.0f, c6 = 1.0f / 720.0f, c5 = 1.0f / 120.0f;
    const float c4 = 1.0f / 24.0f, c3 = 1.0f / 6.0f, c2 = 0.5f;
    float p = c7;
    p = fmaf(p, r, c6);
    p = fmaf(p, r, c5);
    p = fmaf(p, r, c4);
    p = fmaf(p, r, c3);
    p = fmaf(p, r, c2);
    p = fmaf(p, r, 1.0f);
    p = fmaf(p, r, 1.0f);
    return p;
}

float oracle_exp(float y)
{
    if (y < -86.0f) return 0.0f;
    if (y > 88.0f) return INFINITY;
    float n = (y * INV_LN2 + RND) - RND;        /* rint(y / ln 2), ties to even */
    float r = fmaf(-n, LN2_HI, y);              /* n*LN2_HI is exact            */
    r = fmaf(-n, LN2_LO, r);
    return exp_taylor(r) * pow2i((int)n);
}

float oracle_ln(float x)
{
    /* x must be a positive normal number */
    uint32_t i = f2u(x);
    int e = (int)(i >> 23) - 127;
    uint32_t mi = (i & 0x007FFFFFu) | 0x3F800000u;   /* m in [1, 2)  */
    if (mi > 0x3FB504F3u) {                         /* m > sqrt 2   */
        mi -= 0x00800000u;                          /* m / 2        */
        e += 1;
    }
    float m = u2f(mi);
    float f = m - 1.0f;                             /* exact        */
    float s = f / (2.0f + f);
    float z = s * s;
    float q = fmaf(z, 1.0f / 9.0f, 1.0f / 7.0f);
    q = fmaf(z, q, 1.0f / 5.0f);
    q = fmaf(z, q, 1.0f / 3.0f);
    float s2 = s + s;                               /* exact        */
    float lnm = fmaf(s2 * z, q, s2);                /* 2s + 2s z q(z) */
    float ef = (float)e;
    return fmaf(ef, LN2_HI, fmaf(ef, LN2_LO, lnm));
}

float oracle_erfc(float x)
{
    /* x >= 0 */
    if (x == 0.0f) return 1.0f;
    if (!(x < 9.0f)) return 0.0f;
    float t = 1.0f / fmaf(0.5f, x, 1.0f);
    /* g(t) = -1.26551223 + t(1.00002368 + t(0.37409196 + ... + t 0.17087277)) */
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
    /* exp(g - x^2), x^2 = xx + xxl exactly */
    float xx = x * x;
    float xxl = fmaf(x, x, -xx);
    float n = ((g - xx) * INV_LN2 + RND) - RND;
    float r = fmaf(-n, LN2_HI, -xx);
    r = r + g;
    r = r - xxl;
    r = fmaf(-n, LN2_LO, r);
    return t * (exp_taylor(r) * pow2i((int)n));
}

/* r^gamma for r in [0, 1] */
float oracle_pow01(float r, float gamma)
{
    if (r == 0.0f) return 0.0f;
    if (r == 1.0f || gamma == 1.0f) return r;
    return oracle_exp(gamma * oracle_ln(r));
}

/* Eq. 1: survival of the log-normal at dt >= 1; c = fl(1 / fl(sigma * sqrt 2)) */
float oracle_p_lognormal(int32_t dt, float mu, float c)
{
    float u = (oracle_ln((float)dt) - mu) * c;
    if (u >= 0.0f) return 0.5f * oracle_erfc(u);
    return 1.0f - 0.5f * oracle_erfc(-u);
}

/* Eq. 2: position decay; o_b > o_max is treated as r = 1 (caller flags it) */
float oracle_p_structural(int32_t ob, int32_t omax, float gamma)
{
    float r;
    if (omax == 0) r = 0.0f;
    else if (ob >= omax) r = 1.0f;
    else r = (float)ob / (float)omax;
    return 1.0f - oracle_pow01(r, gamma);
}

float oracle_inv_sigma_sqrt2(float sigma) { return 1.0f / (sigma * SQRT2); }

/* Queue kinds (data, per queue) */
enum { K_EVICT_FIRST = 0, K_STRUCTURAL = 1, K_LOGNORMAL = 2, K_RECENCY = 3 };

/*
 * Score n blocks.  Inputs are unpacked per-block fields; theta holds, per
 * queue q < 8: kind[q], alpha[q], mu[q], sigma[q]; w[5]; gamma.
 * Output: key[i] = IEEE bits of P(b) (or of (float)num_tokens for an
 * evict-first queue), and p_out[i] = p_q(b) (Eq. 1 / 2; 1 for recency).
 */
void oracle_score_blocks(int64_t n, int32_t now,
                         const int32_t *last_access, const int32_t *queue,
                         const int32_t *tau, const int32_t *ntok,
                         const int32_t *ob, const int32_t *omax,
                         const int32_t *kind, const float *alpha,
                         const float *mu, const float *sigma,
                         const float *w, float gamma,
                         uint32_t *key, float *p_out)
{
    for (int64_t i = 0; i < n; ++i) {
        int q = queue[i];
        int32_t dt = now - last_access[i];
        if (dt < 0) dt = 0;
        float p;
        if (kind[q] == K_EVICT_FIRST) {
            key[i] = f2u((float)ntok[i]);
            p_out[i] = 1.0f;
            continue;
        } else if (kind[q] == K_LOGNORMAL) {
            p = (dt == 0) ? 1.0f
                          : oracle_p_lognormal(dt, mu[q], oracle_inv_sigma_sqrt2(sigma[q]));
        } else if (kind[q] == K_STRUCTURAL) {
            p = oracle_p_structural(ob[i], omax[i], gamma);
        } else {
            p = 1.0f;
        }
        float aw = alpha[q] * w[tau[i]];
        float nn = aw * p;
        float P = (dt == 0) ? INFINITY : nn / (float)dt;
        key[i] = f2u(P);
        p_out[i] = p;
    }
}

/* element-wise helpers for the pins */
void oracle_ln_v(int64_t n, const float *x, float *y)   { for (int64_t i = 0; i < n; ++i) y[i] = oracle_ln(x[i]); }
void oracle_exp_v(int64_t n, const float *x, float *y)  { for (int64_t i = 0; i < n; ++i) y[i] = oracle_exp(x[i]); }
void oracle_erfc_v(int64_t n, const float *x, float *y) { for (int64_t i = 0; i < n; ++i) y[i] = oracle_erfc(x[i]); }
void oracle_pow01_v(int64_t n, const float *r, float g, float *y) { for (int64_t i = 0; i < n; ++i) y[i] = oracle_pow01(r[i], g); }
void oracle_p_lognormal_v(int64_t n, const int32_t *dt, float mu, float sigma, float *y)
{
    float c = oracle_inv_sigma_sqrt2(sigma);
    for (int64_t i = 0; i < n; ++i) y[i] = (dt[i] == 0) ? 1.0f : oracle_p_lognormal(dt[i], mu, c);
}
void oracle_p_structural_v(int64_t n, const int32_t *ob, const int32_t *omax, float gamma, float *y)
{
    for (int64_t i = 0; i < n; ++i) y[i] = oracle_p_structural(ob[i], omax[i], gamma);
}
