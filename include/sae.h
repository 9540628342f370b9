/*
 * sae.h — C ABI of the MI355X (gfx950) hot path of SAECache's semantic-aware
 * eviction for LLM prefix (KV-block) caches.
 *
 * Paper: "Not All Tokens Are Worth Caching: Learning Semantic-Aware Eviction
 * for LLM Prefix Caches" (arXiv 2605.18825).  Section references below are to
 * that paper.
 *
 * Conventions
 *  - Every call returns sae_status (0 = SAE_OK, negative = error) and never
 *    throws.  Argument validation is synchronous, happens before any launch
 *    and has no side effect on failure; sae_last_error() gives the message.
 *  - Pointers documented "device" are caller-owned device memory (e.g. torch
 *    tensors); they must stay alive until the stream reaches the call.
 *    Pointers documented "host" are read or written before the call returns.
 *  - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL is the
 *    null stream).  A context is not thread-safe: use it from one stream at a
 *    time.  Calls that overlap on one context race, with one exception: a
 *    read-only sae_prefix_match (no flags) may run on another stream while a
 *    sae_score_select without SAE_SS_COMMIT runs, since neither writes what
 *    the other reads (the pool, the index, the parameters).
 *  - The context allocates all of its internal device memory in sae_create();
 *    the hot calls (sae_prefix_match, sae_score_select, sae_match_select,
 *    sae_feedback_update) never allocate.
 *  - Conditions found on the device (index full, o_b > o_max, a slot reused
 *    while still valid, last_access in the future, ...) set bits of a device
 *    status word, read by sae_poll_status().
 *
 * Instances
 *  A context holds n_instances independent caches of blocks_per_instance
 *  blocks each.  Block ids are instance-local, 0 .. blocks_per_instance-1;
 *  per-block arrays are [n_instances * blocks_per_instance], instance-major.
 *
 * Per-block layout (structure of arrays, 10 bytes read by the scoring pass)
 *  last_access  int32  time of last access in ticks (the configurations use
 *                      1 tick = 1 ms); dt = max(now - last_access, 0)
 *  meta         uint16 bit 0-2  queue q (< n_queues)
 *                      bit 3-5  token type tau (SAE_TYPE_*), Sec. 3.1
 *                      bit 6    valid   (block holds cached KV)
 *                      bit 7    leaf    (no cached child block)
 *                      bit 8    ref     (referenced by a running request)
 *                      bit 9-12 num_tokens - 1 (Algorithm 1, stage 1 key)
 *  off          uint32 bit 0-15 o_b, bit 16-31 o_max: block offset and the
 *                      maximum offset in its request (Eq. 2)
 *  hash         uint64 chained content hash; 0 and 2^64-1 are reserved (they
 *                      mark empty and deleted index slots): a block with one is
 *                      refused by Add() and never indexed, and a request hash
 *                      with one never matches
 *  parent       int32  parent block id in the prefix tree, or -1
 *  child_count  int32  number of cached children
 *  ref_count    int32  number of running requests using the block
 *  access_count int32  number of prefix-match hits
 *  The library maintains valid/leaf/ref, child_count, access_count and
 *  last_access (touch) as its calls change them.  meta must be 4-byte
 *  aligned (bits are updated with 32-bit atomics).
 */
#ifndef SAE_H
#define SAE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sae_ctx sae_ctx;
typedef int32_t sae_status;
typedef void *sae_stream_t; /* hipStream_t */

enum {
    SAE_OK = 0,
    SAE_ERR_ARG = -1,   /* invalid argument; nothing was enqueued            */
    SAE_ERR_ALLOC = -2, /* device allocation failed in sae_create            */
    SAE_ERR_HIP = -3,   /* a HIP runtime call failed (message has the error) */
    SAE_ERR_STATE = -4  /* call not valid in the context's state (no pool)   */
};

/* Queue kinds (Sec. 3.1, queue routing; the kind of each queue is data). */
enum {
    SAE_KIND_EVICT_FIRST = 0, /* drained first by num_tokens (Algorithm 1, stage 1) */
    SAE_KIND_STRUCTURAL = 1,  /* position decay, Eq. 2                              */
    SAE_KIND_LOGNORMAL = 2,   /* log-normal survival, Eq. 1 (chat / agentic)        */
    SAE_KIND_RECENCY = 3      /* p = 1: token-weighted recency                      */
};

/* Token types, in the order of Algorithm 3. */
enum {
    SAE_TYPE_SYSTEM = 0,
    SAE_TYPE_USER = 1,
    SAE_TYPE_TOOL = 2,
    SAE_TYPE_RESPONSE = 3,
    SAE_TYPE_COT = 4,
    SAE_N_TYPES = 5
};

#define SAE_MAX_QUEUES 8
#define SAE_N_BINS 8        /* positional bins of the decay-power learner (App. B)      */
#define SAE_IVL_CAP 4096    /* intervals an Algorithm 4 buffer holds between updates    */

#define SAE_META_QUEUE_SHIFT 0
#define SAE_META_TYPE_SHIFT 3
#define SAE_META_VALID 0x0040u
#define SAE_META_LEAF 0x0080u
#define SAE_META_REF 0x0100u
#define SAE_META_NTOK_SHIFT 9

/* Device status bits (sae_poll_status). */
enum {
    SAE_ST_INDEX_FULL = 1u << 0,      /* an index insert found no free slot          */
    SAE_ST_GHOST_FULL = 1u << 1,      /* a recently-evicted insert found no slot     */
    SAE_ST_BAD_OFFSET = 1u << 2,      /* o_b > o_max (scored as o_b = o_max)         */
    SAE_ST_FUTURE_ACCESS = 1u << 3,   /* last_access > now (scored as dt = 0)        */
    SAE_ST_SLOT_BUSY = 1u << 4,       /* insert into a valid slot (insert skipped)   */
    SAE_ST_SELECT_FALLBACK = 1u << 5, /* exact slow path of the pool scan was used   */
    SAE_ST_BAD_BLOCK = 1u << 6,       /* block id out of range (element skipped)     */
    SAE_ST_BAD_HASH = 1u << 7         /* a reserved hash (0 or 2^64-1) given to Add()
                                         or found in a valid block by the index build:
                                         that block is skipped (not added, not indexed) */
};

typedef struct {
    int32_t n_instances;               /* >= 1                                         */
    int32_t blocks_per_instance;       /* >= 1, <= 2^24                               */
    int32_t n_queues;                  /* 1 .. 8                                       */
    int32_t queue_kind[SAE_MAX_QUEUES];/* SAE_KIND_*; at most one evict-first queue    */
    int32_t max_k;                     /* largest k of sae_score_select, 1 .. 8192     */
    int32_t ghost_window;              /* W of recently_evicted (>= 1; 0 = blocks)     */
    int32_t index_log2;                /* index slots per instance = 2^index_log2
                                          (0 = smallest power of two >= 2 blocks)      */
    int32_t max_requests;              /* largest n_req of a sae_prefix_match call with
                                          SAE_PM_INTERVALS, 0 .. 2^24 (0: none)         */
} sae_config;

/* Learned parameters and learner settings (Sec. 3.1, App. B). */
typedef struct {
    float w[SAE_N_TYPES];          /* token-type weights w_tau (Eq. 3)              */
    float alpha[SAE_MAX_QUEUES];   /* queue weights alpha_q (Eq. 3)                 */
    float mu[SAE_MAX_QUEUES];      /* log-normal mu_q, in ln(ticks) (Eq. 1)          */
    float sigma[SAE_MAX_QUEUES];   /* log-normal sigma_q > 0 (Eq. 1)                 */
    float gamma;                   /* position decay power > 0 (Eq. 2)              */
    float eta;                     /* token-weight learning rate (Algorithm 3)      */
    float temperature;             /* T of Algorithm 2, > 0                         */
    float beta;                    /* EMA factor of Algorithm 2 and of gamma        */
    float beta_ln;                 /* EMA factor of Algorithm 4 (beta_ln)           */
    int32_t K;                     /* learners run every K evictions (Algorithm 1)  */
    uint32_t learn;                /* SAE_LEARN_* bits                              */
} sae_params;

enum {
    SAE_LEARN_TOKEN_WEIGHTS = 1u << 0, /* Algorithm 3                              */
    SAE_LEARN_QUEUE_WEIGHTS = 1u << 1, /* Algorithm 2                              */
    SAE_LEARN_LOGNORMAL = 1u << 2,     /* Algorithm 4: mu_q, sigma_q              */
    SAE_LEARN_DECAY_POWER = 1u << 3,   /* gamma from positional hit rates (App. B) */
    SAE_LEARN_TOKEN_EMA = 1u << 4,     /* App. B text's token-weight rule; replaces
                                          Algorithm 3 (not both)                   */
    SAE_LEARN_QUEUE_REL = 1u << 5      /* App. B text's queue-weight rule; replaces
                                          Algorithm 2 (not both)                   */
};

/* Feedback counters of one instance (Algorithms 1-3). */
typedef struct {
    int32_t evicted[SAE_N_TYPES];     /* token_stats[tau].evicted                 */
    int32_t missed[SAE_N_TYPES];      /* token_stats[tau].miss_after_evict        */
    int32_t hits[SAE_MAX_QUEUES];     /* queue_hits[q]                            */
    int32_t evictions[SAE_MAX_QUEUES];/* queue_evictions[q]                       */
    int64_t eviction_count;           /* all evictions so far                     */
    int32_t pending;                  /* learners due (eviction_count crossed K)  */
    int32_t n_updates;                /* learner runs so far                      */
    int32_t bin_hits[SAE_N_BINS];     /* decay-power learner: prefix-match hits of
                                         structural blocks per positional bin     */
    int32_t bin_missed[SAE_N_BINS];   /* ... and misses after their eviction
                                         (both only while SAE_LEARN_DECAY_POWER) */
    int32_t type_hits[SAE_N_TYPES];   /* SAE_LEARN_TOKEN_EMA: prefix-match hits per
                                         block type ...                           */
    int32_t type_added[SAE_N_TYPES];  /* ... and blocks added per type (Add())    */
    int32_t resident[SAE_MAX_QUEUES]; /* cached (valid) blocks per queue          */
} sae_counters;

/* Caller-owned device arrays of the block pool (layout above). */
typedef struct {
    int32_t *last_access;
    uint16_t *meta;
    uint32_t *off;
    uint64_t *hash;
    int32_t *parent;
    int32_t *child_count;
    int32_t *ref_count;
    int32_t *access_count;
} sae_pool;

const char *sae_status_str(sae_status s);
/* Last error message of ctx (or of the last failed sae_create when ctx is NULL). */
const char *sae_last_error(const sae_ctx *ctx);

/* Create a context and allocate all of its device memory on the current
 * device: index, recently-evicted table, per-instance parameters and counters,
 * selection scratch.  *out is set only on success. */
sae_status sae_create(const sae_config *cfg, sae_ctx **out);
sae_status sae_destroy(sae_ctx *ctx);

/* Attach the caller's pool arrays (all required, device, sized
 * n_instances * blocks_per_instance).  Does not read them. */
sae_status sae_bind_pool(sae_ctx *ctx, const sae_pool *pool);

/* Parameters of one instance (inst >= 0) or of all (inst = -1); host struct
 * copied before return.  sigma, gamma, temperature must be > 0; at most one
 * token-weight rule and one queue-weight rule may be chosen in `learn`. */
sae_status sae_set_params(sae_ctx *ctx, int32_t inst, const sae_params *p, sae_stream_t stream);
/* Read back parameters / counters of one instance; synchronizes `stream`. */
sae_status sae_get_params(sae_ctx *ctx, int32_t inst, sae_params *out, sae_stream_t stream);
sae_status sae_get_counters(sae_ctx *ctx, int32_t inst, sae_counters *out, sae_stream_t stream);
/* Overwrite one instance's counters (checkpoint / resume). */
sae_status sae_set_counters(sae_ctx *ctx, int32_t inst, const sae_counters *c, sae_stream_t stream);

/* Block type tau(b) = type of the block's median token (Sec. 3.1), from
 * per-block token-type counts: counts[n][5] uint8 (device), tau[n] uint8
 * (device).  Tokens are ranked by type in SAE_TYPE order; the median is the
 * lower median (rank floor((n_tokens - 1) / 2)). */
sae_status sae_block_type(const uint8_t *counts, int64_t n, uint8_t *tau, sae_stream_t stream);

/* Cache hints of a block (one byte each), the input of Algorithm 1's Classify. */
enum {
    SAE_HINT_DECODE = 1u << 0,        /* holds decode-phase (generated) tokens                 */
    SAE_HINT_UNTEMPLATED = 1u << 1,   /* prefill content outside any shared template          */
    SAE_HINT_MULTI_TURN = 1u << 2,    /* its request is (or is predicted to be) multi-turn    */
    SAE_HINT_AGENTIC = 1u << 3,       /* its request is agentic / tool use                    */
    SAE_HINT_CONVERSATION = 1u << 4,  /* its request carries a conversation id (has history)  */
    SAE_HINT_SHARED_PREFIX = 1u << 5  /* lies in a prompt template shared across requests     */
};
/* Queues that Classify routes to: roles[SAE_ROLE_*] is a queue index. */
enum { SAE_ROLE_EVICT = 0, SAE_ROLE_STRUCT = 1, SAE_ROLE_CHAT = 2, SAE_ROLE_AGENT = 3, SAE_N_ROLES = 4 };

/*
 * Algorithm 1 Classify (queue routing, Sec. 3.1): for n blocks, from the hint
 * byte and the block type tau already in meta, the first rule that holds:
 *   tau = cot, or decode, or untemplated  -> evict-first
 *   multi-turn and agentic                -> agent
 *   multi-turn, or conversation           -> chat
 *   shared prefix, or tau = system        -> structural
 *   otherwise                             -> evict-first
 *  hint[n]   device uint8
 *  meta[n]   device uint16, in/out: the queue bits are replaced by
 *            roles[rule] (the other bits are kept)
 *  roles[4]  host int32 queue indices, each in 0 .. n_queues-1
 * Returns SAE_ERR_ARG (nothing launched) for a bad role or a NULL array.
 */
sae_status sae_classify_blocks(sae_ctx *ctx, int32_t n, const uint8_t *hint, uint16_t *meta,
                               const int32_t *roles, sae_stream_t stream);

/* Rebuild the block index (content hash -> block) from the hash of every
 * valid block, and clear recently_evicted and all counters.  Use after
 * filling the pool arrays directly.  Hashes of valid blocks must be distinct
 * within an instance. */
sae_status sae_index_build(sae_ctx *ctx, sae_stream_t stream);

/*
 * Algorithm 1, Add(b, h), for a batch of n new blocks placed in free slots.
 *  inst[n]   device int32 instance of each block, or NULL (all instance 0)
 *  ids[n]    device int32 instance-local block id (slot must not be valid)
 *  hash[n], parent[n] (-1 = root), last_access[n]: device
 *  meta[n]   device uint16: queue, type and num_tokens fields are used; the
 *            library sets valid and leaf, clears ref
 *  off[n]    device uint32 (o_b, o_max)
 * Each block goes into the index.  A hash still in recently_evicted counts
 * one miss after eviction for the type recorded at eviction (Algorithm 1,
 * Add; Algorithm 3's miss_after_evict) and leaves recently_evicted.  Parents
 * gain a child (and lose their leaf bit).  Hashes must be distinct and absent
 * from the index.  Busy slots set SAE_ST_SLOT_BUSY and are skipped.
 */
sae_status sae_insert_blocks(sae_ctx *ctx, int32_t n, const int32_t *inst, const int32_t *ids,
                             const uint64_t *hash, const int32_t *parent, const int32_t *last_access,
                             const uint16_t *meta, const uint32_t *off, sae_stream_t stream);

/* ref_count[b] += delta for n blocks (device inst[n] or NULL, ids[n]); the ref
 * bit of meta follows ref_count > 0.  A referenced block is not evictable. */
sae_status sae_ref_blocks(sae_ctx *ctx, int32_t n, const int32_t *inst, const int32_t *ids,
                          int32_t delta, sae_stream_t stream);

/* Flags of sae_prefix_match */
enum { SAE_PM_TOUCH = 1u << 0, SAE_PM_STATS = 1u << 1, SAE_PM_INTERVALS = 1u << 2 };

/*
 * HOT 1 — batched strict prefix matching (Sec. 2.1: a later block is reusable
 * only if every earlier block matches; blocks are identified by content hash).
 *  hashes[n_req][max_len]  device uint64, request r's block hashes in order
 *  lens[n_req]             device int32, 0 <= lens[r] <= max_len
 *  inst[n_req]             device int32 or NULL (instance 0)
 *  match_len[n_req]        device int32 out: number of leading hashes present
 *                          in the index (the first miss ends the match)
 *  matched_ids             device int32 [n_req][max_len] out or NULL: block id
 *                          of each matched position, -1 elsewhere
 * Every request sees the index as it was before the call.  SAE_PM_TOUCH sets
 * last_access = now and adds 1 to access_count for every (request, matched
 * block); SAE_PM_STATS adds every matched block to queue_hits[its queue]
 * (Algorithm 2) and, in a structural queue of an instance whose
 * SAE_LEARN_DECAY_POWER bit is set, to the hits of its positional bin
 * floor(8 o_b / o_max) (decay-power learner, App. B); with SAE_LEARN_TOKEN_EMA
 * set, to type_hits[its type].
 * The queue, type and positional bin counted for a block are the ones it had
 * when it entered the index (sae_insert_blocks or sae_index_build): a caller
 * that rewrites those pool fields of a valid block rebuilds the index.
 * SAE_PM_INTERVALS records Algorithm 4's reuse intervals: for every request
 * and every log-normal queue among its matched blocks, dt = now - last_access
 * of its deepest matched block of that queue, as it was before the call,
 * if 1 <= dt < 2^31; a call's intervals join that queue's buffer in request
 * order (the buffer keeps the newest SAE_IVL_CAP).  It needs matched_ids
 * (the touch pass reads it) and n_req <= sae_config.max_requests.
 * Without TOUCH, STATS and INTERVALS the call is read-only.
 */
sae_status sae_prefix_match(sae_ctx *ctx, int32_t n_req, int32_t max_len, const uint64_t *hashes,
                            const int32_t *lens, const int32_t *inst, int32_t now, uint32_t flags,
                            int32_t *match_len, int32_t *matched_ids, sae_stream_t stream);

/* Flags of sae_score_select */
enum {
    SAE_SS_COMMIT = 1u << 0,          /* evict the decision (see below)                  */
    SAE_SS_ENGINE_SCAN = 1u << 1,     /* force the pool-scan engine                      */
    SAE_SS_ENGINE_BATCHED = 1u << 2,  /* force the one-workgroup-per-instance engine     */
    SAE_SS_FORCE_FALLBACK = 1u << 3,  /* pool-scan engine: take its exact slow path      */
    SAE_SS_CASCADE = 1u << 4          /* decision: Algorithm 1 one victim at a time      */
};

/*
 * HOT 2 — score every block and select victims.
 * Score (Sec. 3.1): dt = max(now - last_access, 0);
 *   p_q(b) = 1 - F_LN(dt; mu_q, sigma_q)       log-normal queues (Eq. 1)
 *          = 1 - (o_b / o_max)^gamma           structural queues (Eq. 2)
 *          = 1                                 recency queues
 *   P(b)   = alpha_q w_tau(b) p_q(b) / dt      (Eq. 3; dt = 0 gives +inf)
 * evaluated in a fixed fp32 recipe (IEEE + - * /, fma, exact bit operations).
 * An evict-first queue is ordered by num_tokens (Algorithm 1, stage 1).
 * A block is evictable iff valid, leaf and unreferenced.
 * Select: for every instance i and queue q, the c = min(k_i, #evictable in q)
 * evictable blocks with the smallest (key, block id), ascending:
 *   victims[i][q][0..c)  device int32, stride max_k per queue
 *   scores[i][q][0..c)   device float (P, or num_tokens for evict-first) or NULL
 *   count[i][q]          device int32
 * Decision (Algorithm 1 applied k_i times to this snapshot): the evict-first
 * list first, then the other queues merged by (P, id):
 *   decision[i][0..d)    device int32, stride max_k;  decision_count[i] = d
 * k_i = k_per_inst[i] (device int32, or NULL for k); 0 <= k_i <= max_k.
 * SAE_SS_COMMIT then evicts the decision: valid bit cleared, index entry
 * removed, hash -> (tau, queue) recorded in recently_evicted, evicted[tau] and
 * queue_evictions[q] incremented, parent's child_count decremented (a parent
 * left with no child becomes a leaf, eligible from the next call), and the
 * learners are marked due when eviction_count crosses a multiple of K.
 * Ties are broken by block id.  Results do not depend on the engine.
 * SAE_SS_CASCADE makes the decision the one of k successive Evict() calls on
 * the live state (Algorithm 1 as printed): a parent whose last cached child
 * is taken becomes a leaf, evictable by the next call, so a decision can hold
 * a block together with its ancestors.  Needs max_k <= 4096; the per-queue
 * lists stay the snapshot's.
 */
sae_status sae_score_select(sae_ctx *ctx, int32_t now, int32_t k, const int32_t *k_per_inst,
                            uint32_t flags, int32_t *victims, float *scores, int32_t *count,
                            int32_t *decision, int32_t *decision_count, sae_stream_t stream);

/*
 * HOT 1 + HOT 2 — a serving step's prefix match and eviction as one call
 * (Sec. 2.1, then Sec. 3.1 and Algorithm 1 on the pool the match left).
 * Same arguments, checks, errors and results as sae_prefix_match(ctx, n_req,
 * max_len, hashes, lens, inst, pm_now, pm_flags, match_len, matched_ids)
 * followed on the same stream by sae_score_select(ctx, now, k, k_per_inst,
 * flags, victims, scores, count, decision, decision_count): every output,
 * and every change to the pool, index and counters, is the one of those two
 * calls in that order.  With the pool-scan engine the selection's sample of
 * the pool and its per-queue candidate bounds are computed in the prefix
 * match's launch, while the requests probe the index, so the step has two
 * launches fewer on its critical path.  A sampled block may be seen before
 * or after the match touches it; the bounds only steer the work (the exact
 * path takes over wherever they would miss a victim, SAE_ST_SELECT_FALLBACK),
 * so no result depends on it.  An argument error of either half fails the
 * whole call before anything is enqueued.
 */
sae_status sae_match_select(sae_ctx *ctx, int32_t n_req, int32_t max_len, const uint64_t *hashes,
                            const int32_t *lens, const int32_t *inst, int32_t pm_now, uint32_t pm_flags,
                            int32_t *match_len, int32_t *matched_ids, int32_t now, int32_t k,
                            const int32_t *k_per_inst, uint32_t flags, int32_t *victims, float *scores,
                            int32_t *count, int32_t *decision, int32_t *decision_count,
                            sae_stream_t stream);

/* Flags of sae_feedback_update */
enum { SAE_FB_FORCE = 1u << 0 };

/*
 * HOT 3 — eviction-feedback learners of every instance whose learners are due
 * (or all with SAE_FB_FORCE), in fp32:
 *  Algorithm 3 (token weights): for each tau with evicted > 10,
 *    w_tau <- clamp(w_tau * (1 + eta * missed / evicted), 0.1, 5.0);
 *    then evicted <- floor(0.99 evicted), missed <- floor(0.99 missed)
 *    (0.99 applied exactly as 99/100).
 *  Algorithm 2 (queue weights): for each queue but the evict-first one with
 *    evictions > 5, alpha_q <- clamp(alpha_q + beta (1 + (hits/evictions)/T
 *    - alpha_q), 0.1, 3.0); then hits and evictions reset to 0.
 *  Algorithm 4 (log-normal parameters): for each log-normal queue whose
 *    interval buffer holds n > 20 intervals: with x = ln dt (the fp32 recipe's
 *    ln), mu_s = mean x, sigma_s = population std of x (exact integer sums of
 *    x * 2^24, then rounded in double and to fp32),
 *    mu_q <- mu_q + beta_ln (mu_s - mu_q), sigma_q <- max(sigma_q +
 *    beta_ln (sigma_s - sigma_q), 0.1); the buffer keeps its last 200.
 *  Decay power (App. B): with rate_i = hits_i / (hits_i + missed_i) over the
 *    bins that had events, front = mean rate of bins 0-3, back = of bins 4-7;
 *    if there were more than 20 events, both halves had some and front > 0:
 *    gamma <- clamp(gamma + beta (1 / (back / front + 0.1) - gamma), 0.3, 3.0)
 *    and the bin counters restart.
 *  Token weights, the appendix text's rule (SAE_LEARN_TOKEN_EMA): for every
 *    type, w_target = 1 + 5 r_miss + 2 r_reuse with r_miss = missed / evicted
 *    and r_reuse = type_hits / (type_hits + type_added) (0 when undefined),
 *    w <- clamp((1 - eta) w + eta w_target, 0.1, 5.0); the four counters decay
 *    as floor(0.99 x).
 *  Queue weights, the appendix text's rule (SAE_LEARN_QUEUE_REL): over the
 *    queues but the evict-first one that hold blocks, E_q = hits_q /
 *    (resident_q / resident_all), E_mean their mean; if E_mean > 0,
 *    alpha_q <- clamp(beta alpha_q + (1 - beta) (E_q / E_mean)^(1/T), 0.1, 3.0)
 *    (the power as the fp32 recipe's exp(ln x / T), x itself for T = 1); hits
 *    and evictions then reset.
 * Each algorithm runs only if its SAE_LEARN_* bit is set.
 */
sae_status sae_feedback_update(sae_ctx *ctx, uint32_t flags, sae_stream_t stream);

/*
 * Checkpoint and resume of one instance's state held by the context: its
 * learned parameters and learner settings, every feedback counter, the
 * eviction count, Algorithm 4's interval buffers and the recently_evicted
 * ring (Algorithm 1), as one opaque blob.  The pool arrays are the caller's;
 * the block index is rebuilt from them.
 *  sae_state_size:  *bytes (host) = the blob size for this context's shape
 *  sae_save_state:  writes the blob of instance `inst` to buf (host, `bytes`
 *                   = sae_state_size) and synchronizes `stream`
 *  sae_load_state:  restores instance `inst` from a blob saved by a context
 *                   of the same shape (queues and kinds, max_k, ghost window,
 *                   blocks per instance); SAE_ERR_ARG (nothing changed) for a
 *                   blob of another shape or size.  It rebuilds the
 *                   recently_evicted table and synchronizes `stream`.
 * To resume: copy the pool arrays, sae_create a context of the same shape,
 * sae_bind_pool, sae_index_build (which clears state), then sae_load_state
 * for every instance.  The resumed instance then decides, matches and
 * learns exactly as the saved one would have.
 */
sae_status sae_state_size(sae_ctx *ctx, size_t *bytes);
sae_status sae_save_state(sae_ctx *ctx, int32_t inst, void *buf, size_t bytes, sae_stream_t stream);
sae_status sae_load_state(sae_ctx *ctx, int32_t inst, const void *buf, size_t bytes, sae_stream_t stream);

/* Algorithm 4's interval buffer of one (instance, log-normal queue), oldest
 * first: out (host int32, cap entries) receives the first min(n, cap)
 * intervals in ticks and *n (host) the number held.  Synchronizes `stream`.
 * SAE_ERR_ARG for a queue that is not log-normal. */
sae_status sae_get_intervals(sae_ctx *ctx, int32_t inst, int32_t queue, int32_t *out, int32_t cap, int32_t *n,
                             sae_stream_t stream);

/* OR of the device status bits since the last poll (then cleared);
 * synchronizes `stream`. */
sae_status sae_poll_status(sae_ctx *ctx, sae_stream_t stream, uint32_t *bits);

/* Diagnostics of the last pool-scan selection of one instance: for each
 * queue q, out[4q..4q+3] = {evictable blocks (0xFFFFFFFF when the selection
 * did not need the count: the bound admitted only part of the queue and the
 * exact slow path did not run), candidates under the bound that were kept,
 * candidates beyond the capacity of the candidate stripes (they send the
 * selection to the exact slow path), 1 if the exact slow path ran}.  out is
 * host memory of 4 * n_queues words; synchronizes `stream`. */
sae_status sae_select_stats(sae_ctx *ctx, int32_t inst, uint32_t *out, sae_stream_t stream);

/*
 * Multi-turn session predictor (Sec. 3.3): for each request, the serving
 * model's final-layer hidden state h of its last prompt token goes through
 *   y = W3 relu(W2 relu(W1 h + b1) + b2) + b3
 * (hidden widths 256 and 64); y > 0 predicts that the session continues.
 *  h[n][d]       device bf16 (uint16 bit patterns), row-major
 *  w->w1[256][d] device bf16, row-major (one row per first-layer unit)
 *  w->b1[256], w->w2[64][256] (row-major), w->b2[64], w->w3[64], w->b3[1]
 *                device float
 *  work[4][n][256] device float scratch (the first layer's partial sums)
 *  logit[n]      device float out: y
 *  pred[n]       device uint8 out: 1 if y > 0, else 0 (or NULL)
 * Layer 1 multiplies bf16 exactly and sums in fp32 (matrix cores), in four k
 * slices added in a fixed order; layers 2 and 3 are fp32.  Needs
 * 256 <= d <= 16384 with d a multiple of 256, n >= 0.
 * Returns SAE_ERR_ARG (nothing launched) otherwise or for a NULL array.
 */
#define SAE_PRED_H1 256
#define SAE_PRED_H2 64
typedef struct {
    const uint16_t *w1;
    const float *b1;
    const float *w2;
    const float *b2;
    const float *w3;
    const float *b3;
} sae_predictor;
sae_status sae_predict_sessions(int32_t n, int32_t d, const uint16_t *h, const sae_predictor *w, float *work,
                                float *logit, uint8_t *pred, sae_stream_t stream);

/*
 * Session predictor for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same computation and results as sae_predict_sessions, with
 * no `work` argument.  Layer 1's partial sums go to a buffer of the library's
 * own, one per GPU, of SAE_PRED_NOALLOC_MAX_N rows (16 MiB), held by each GPU
 * the library runs on until the process ends; the call allocates nothing.
 * Every call on a GPU shares that buffer, so calls that overlap on one GPU
 * (several streams, threads or processes' contexts in flight at once) race;
 * calls in stream order do not.  Nothing in the buffer needs to start at zero:
 * every partial sum read is written first by the same call.
 * SAE_ERR_ARG (nothing launched) for n > SAE_PRED_NOALLOC_MAX_N and the
 * conditions of sae_predict_sessions.
 */
#define SAE_PRED_NOALLOC_MAX_N 4096
sae_status sae_predict_sessions_noalloc(int32_t n, int32_t d, const uint16_t *h, const sae_predictor *w,
                                        float *logit, uint8_t *pred, sae_stream_t stream);

/* Device realisation of the fp32 recipe's elementary functions (the ones
 * Eq. 1 and Eq. 2 are built from), element-wise, for checking it:
 *  fn = SAE_FN_LN    y = ln x    (x a positive normal float)
 *       SAE_FN_EXP   y = e^x
 *       SAE_FN_ERFC  y = erfc x  (x >= 0)
 *  x[n], y[n] device float.  Returns SAE_ERR_ARG for an unknown fn, n < 0 or
 *  a NULL array with n > 0 (nothing launched). */
enum { SAE_FN_LN = 0, SAE_FN_EXP = 1, SAE_FN_ERFC = 2 };
sae_status sae_recipe_eval(int32_t fn, int64_t n, const float *x, float *y, sae_stream_t stream);

/* Per-kernel timing of the pool-scan engine's scoring pass: when enabled,
 * every launch of that kernel carries a pair of HIP events that record the
 * dispatch's own start and end on the call's stream.
 * sae_profile_read returns the summed milliseconds and launch count since the
 * last read (synchronizes) and resets them. */
sae_status sae_profile_enable(sae_ctx *ctx, int32_t enable);
sae_status sae_profile_read(sae_ctx *ctx, double *ms, int64_t *launches);

#ifdef __cplusplus
}
#endif
#endif /* SAE_H */
