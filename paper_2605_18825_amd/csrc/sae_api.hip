// C ABI of libsae: context lifetime, argument validation and launch
// sequencing.  No call allocates device memory after sae_create.
#include <stddef.h>
#include <stdio.h>
#include <string.h>

#include <string>
#include <utility>
#include <vector>

#include "sae_internal.h"

struct sae_ctx {
    sae_config cfg;
    DevCtx dc;
    bool pool_bound = false;
    int device = 0;
    std::string err;
    long long index_slots = 0, ghost_slots = 0;
    double index_tombs = 0, ghost_tombs = 0;
    uint8_t *skip = nullptr;
    long long skip_cap = 0;
    std::vector<void *> allocs;
    bool prof = false;
    int casc_set = 0;  // the counter set the next cascading decision uses
    uint32_t prep_calls = 0;  // pool-scan sae_match_select calls so far (wraps)
    std::vector<std::pair<hipEvent_t, hipEvent_t>> prof_used;
    std::vector<std::pair<hipEvent_t, hipEvent_t>> prof_free;
};

namespace {

thread_local std::string g_err;

sae_status fail(sae_ctx *c, sae_status s, const std::string &msg)
{
    if (c) c->err = msg;
    else g_err = msg;
    return s;
}

sae_status hip_fail(sae_ctx *c, hipError_t e, const char *what)
{
    std::string m = std::string(what) + ": " + hipGetErrorString(e);
    return fail(c, SAE_ERR_HIP, m);
}

template <typename T>
bool dev_alloc(sae_ctx *c, T **p, size_t count)
{
    size_t bytes = count * sizeof(T);
    if (bytes == 0) bytes = 256;
    void *q = nullptr;
    if (hipMalloc(&q, bytes) != hipSuccess) return false;
    if (hipMemset(q, 0, bytes) != hipSuccess) {
        (void)hipFree(q);
        return false;
    }
    c->allocs.push_back(q);
    *p = static_cast<T *>(q);
    return true;
}

int log2_ceil(long long x)
{
    int l = 0;
    while ((1ll << l) < x) ++l;
    return l;
}

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

void default_params(InstState &s, int max_k)
{
    memset(&s, 0, sizeof(s));
    for (int t = 0; t < SAE_N_TYPES; ++t) s.w[t] = 1.0f;
    for (int q = 0; q < SAE_MAX_QUEUES; ++q) {
        s.alpha[q] = 1.0f;
        s.mu[q] = 0.0f;
        s.sigma[q] = 1.0f;
    }
    s.gamma = 1.0f;
    s.eta = 0.01f;
    s.T = 1.0f;
    s.beta = 0.1f;
    s.beta_ln = 0.1f;
    s.K = max_k;
    s.learn = SAE_LEARN_TOKEN_WEIGHTS | SAE_LEARN_QUEUE_WEIGHTS;
}

hipStream_t S(sae_stream_t s) { return reinterpret_cast<hipStream_t>(s); }

sae_status check_inst(sae_ctx *c, int32_t inst, bool allow_all)
{
    if (inst == -1 && allow_all) return SAE_OK;
    if (inst < 0 || inst >= c->cfg.n_instances) return fail(c, SAE_ERR_ARG, "instance out of range");
    return SAE_OK;
}

}  // namespace

extern "C" {

const char *sae_status_str(sae_status s)
{
    switch (s) {
    case SAE_OK: return "ok";
    case SAE_ERR_ARG: return "invalid argument";
    case SAE_ERR_ALLOC: return "device allocation failed";
    case SAE_ERR_HIP: return "HIP runtime error";
    case SAE_ERR_STATE: return "invalid state";
    default: return "unknown status";
    }
}

const char *sae_last_error(const sae_ctx *ctx) { return ctx ? ctx->err.c_str() : g_err.c_str(); }

sae_status sae_create(const sae_config *cfg, sae_ctx **out)
{
    if (!cfg || !out) return fail(nullptr, SAE_ERR_ARG, "cfg and out must be non-NULL");
    const sae_config &k = *cfg;
    if (k.n_instances < 1 || k.n_instances > 65535) return fail(nullptr, SAE_ERR_ARG, "n_instances must be in 1..65535");
    if (k.blocks_per_instance < 1 || k.blocks_per_instance > (1 << 24))
        return fail(nullptr, SAE_ERR_ARG, "blocks_per_instance must be in 1..2^24");
    if (k.n_queues < 1 || k.n_queues > SAE_MAX_QUEUES) return fail(nullptr, SAE_ERR_ARG, "n_queues must be in 1..8");
    if (k.max_k < 1 || k.max_k > 8192) return fail(nullptr, SAE_ERR_ARG, "max_k must be in 1..8192");
    if (k.ghost_window < 0) return fail(nullptr, SAE_ERR_ARG, "ghost_window must be >= 0");
    if (k.index_log2 < 0 || k.index_log2 > 30) return fail(nullptr, SAE_ERR_ARG, "index_log2 must be in 0..30");
    if (k.max_requests < 0 || k.max_requests > (1 << 24))
        return fail(nullptr, SAE_ERR_ARG, "max_requests must be in 0..2^24");
    int n_ef = 0;
    for (int q = 0; q < k.n_queues; ++q) {
        if (k.queue_kind[q] < SAE_KIND_EVICT_FIRST || k.queue_kind[q] > SAE_KIND_RECENCY)
            return fail(nullptr, SAE_ERR_ARG, "unknown queue kind");
        n_ef += (k.queue_kind[q] == SAE_KIND_EVICT_FIRST);
    }
    if (n_ef > 1) return fail(nullptr, SAE_ERR_ARG, "at most one evict-first queue");

    sae_ctx *c = new sae_ctx();
    c->cfg = k;
    (void)hipGetDevice(&c->device);
    DevCtx &d = c->dc;
    memset(&d, 0, sizeof(d));
    d.n_inst = k.n_instances;
    d.N = k.blocks_per_instance;
    d.Q = k.n_queues;
    if (hipDeviceGetAttribute(&d.n_cu, hipDeviceAttributeMultiprocessorCount, c->device) != hipSuccess || d.n_cu < 1)
        d.n_cu = 1;
    d.max_k = k.max_k;
    d.ef_queue = -1;
    for (int q = 0; q < SAE_MAX_QUEUES; ++q) d.kind[q] = (q < k.n_queues) ? k.queue_kind[q] : SAE_KIND_RECENCY;
    for (int q = 0; q < k.n_queues; ++q) {
        if (k.queue_kind[q] == SAE_KIND_EVICT_FIRST) d.ef_queue = q;
        if (k.queue_kind[q] == SAE_KIND_LOGNORMAL) d.ln_mask |= 1u << q;
        if (k.queue_kind[q] == SAE_KIND_STRUCTURAL) d.struct_mask |= 1u << q;
    }
    d.max_req = k.max_requests;
    d.casc_tl = 8 * k.max_k;
    d.W = k.ghost_window ? k.ghost_window : k.blocks_per_instance;
    d.ring_cap = d.W + d.max_k;
    int il = k.index_log2 ? k.index_log2 : log2_ceil(2ll * d.N);
    if (il < 6) il = 6;
    if ((1ll << il) < (long long)d.N + 1) {
        delete c;
        return fail(nullptr, SAE_ERR_ARG, "index_log2 too small for blocks_per_instance");
    }
    int gl = log2_ceil(2ll * d.ring_cap);
    if (gl < 6) gl = 6;
    c->index_slots = 1ll << il;
    c->ghost_slots = 1ll << gl;
    d.index_mask = (uint32_t)(c->index_slots - 1);
    d.ghost_mask = (uint32_t)(c->ghost_slots - 1);

    const long long I = d.n_inst, Q = d.Q;
    d.scan_gx = scan_grid_x(d.n_inst, d.N);
    bool ok = dev_alloc(c, &d.state, I) && dev_alloc(c, &d.status, 1) &&
              dev_alloc(c, &d.index, I * c->index_slots) && dev_alloc(c, &d.ring, I * d.ring_cap) &&
              dev_alloc(c, &d.gtab, I * c->ghost_slots) && dev_alloc(c, &d.thr, I * Q) && dev_alloc(c, &d.sent, I * 64) && dev_alloc(c, &d.eflim, I * 16) &&
              dev_alloc(c, &d.split, I * Q * SAE_NBUCKET) && dev_alloc(c, &d.nsplit, I * Q) &&
              dev_alloc(c, &d.cand, I * Q * 2 * SAE_LCAP) && dev_alloc(c, &d.stripe_n, I * Q * (SAE_STRIPES + 1)) &&
              dev_alloc(c, &d.cpart, I * SAE_CSLOTS * SAE_CF_STRIDE) &&
              dev_alloc(c, &d.samp, I * SAE_SAMPLE_WGS * SAE_SAMPLE_CHUNK) &&
              dev_alloc(c, &d.samp_qn, I * SAE_SAMPLE_WGS * SAE_MAX_QUEUES) &&
              dev_alloc(c, &d.prep_done, I) &&
              dev_alloc(c, &d.sel, I * Q * d.max_k) && dev_alloc(c, &d.sel_count, I * Q) &&
              dev_alloc(c, &d.sel_stats, I * Q * 4) && dev_alloc(c, &c->skip, I * d.N) &&
              dev_alloc(c, &d.ivl, d.ln_mask ? I * Q * SAE_IVL_CAP : 0) &&
              dev_alloc(c, &d.pm_rec, (long long)d.max_req * SAE_MAX_QUEUES) &&
              dev_alloc(c, &d.casc_cnt, 2 * I * d.N) && dev_alloc(c, &d.casc_e, 2 * I * d.N) &&
              dev_alloc(c, &d.casc_touch, 2 * I * 8ll * d.max_k) && dev_alloc(c, &d.casc_nt, 2 * I) &&
              dev_alloc(c, &d.casc_k0, I * d.max_k) &&
              dev_alloc(c, &d.casc_prom, I * d.max_k) && dev_alloc(c, &d.casc_pe, I * d.max_k) &&
              dev_alloc(c, &d.casc_aid, I * d.max_k) &&
              dev_alloc(c, &d.casc_n, I * 4);
    // the batched engine's key cache, where that engine can run
    const long long nb = batched_engine_fits(d) ? I * d.N : 0;
    ok = ok && dev_alloc(c, &d.bkey, nb) && dev_alloc(c, &d.bq, nb);
    if (!ok) {
        for (void *p : c->allocs) (void)hipFree(p);
        delete c;
        return fail(nullptr, SAE_ERR_ALLOC, "hipMalloc failed in sae_create");
    }
    c->skip_cap = I * d.N;
    std::vector<InstState> init((size_t)I);
    for (auto &s : init) default_params(s, d.max_k);
    hipError_t e = hipMemcpy(d.state, init.data(), sizeof(InstState) * I, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) {
        for (void *p : c->allocs) (void)hipFree(p);
        delete c;
        return hip_fail(nullptr, e, "sae_create init");
    }
    *out = c;
    return SAE_OK;
}

sae_status sae_destroy(sae_ctx *c)
{
    if (!c) return SAE_OK;
    (void)hipDeviceSynchronize();
    for (auto &p : c->prof_used) {
        (void)hipEventDestroy(p.first);
        (void)hipEventDestroy(p.second);
    }
    for (auto &p : c->prof_free) {
        (void)hipEventDestroy(p.first);
        (void)hipEventDestroy(p.second);
    }
    for (void *p : c->allocs) (void)hipFree(p);
    delete c;
    return SAE_OK;
}

sae_status sae_bind_pool(sae_ctx *c, const sae_pool *p)
{
    if (!c || !p) return fail(c, SAE_ERR_ARG, "ctx and pool must be non-NULL");
    if (!p->last_access || !p->meta || !p->off || !p->hash || !p->parent || !p->child_count || !p->ref_count ||
        !p->access_count)
        return fail(c, SAE_ERR_ARG, "every pool array must be non-NULL");
    if (!aligned(p->last_access, 16) || !aligned(p->off, 16) || !aligned(p->meta, 8) || !aligned(p->hash, 8) ||
        !aligned(p->parent, 4) || !aligned(p->child_count, 4) || !aligned(p->ref_count, 4) ||
        !aligned(p->access_count, 4))
        return fail(c, SAE_ERR_ARG, "pool alignment: last_access/off 16 B, meta/hash 8 B, others 4 B");
    DevCtx &d = c->dc;
    d.la = p->last_access;
    d.meta = p->meta;
    d.off = p->off;
    d.hash = reinterpret_cast<unsigned long long *>(p->hash);
    d.parent = p->parent;
    d.child_count = p->child_count;
    d.ref_count = p->ref_count;
    d.access_count = p->access_count;
    c->pool_bound = true;
    return SAE_OK;
}

sae_status sae_set_params(sae_ctx *c, int32_t inst, const sae_params *p, sae_stream_t stream)
{
    if (!c || !p) return fail(c, SAE_ERR_ARG, "ctx and params must be non-NULL");
    if (check_inst(c, inst, true) != SAE_OK) return SAE_ERR_ARG;
    for (int q = 0; q < c->dc.Q; ++q)
        if (!(p->sigma[q] > 0.0f)) return fail(c, SAE_ERR_ARG, "sigma must be > 0");
    if (!(p->gamma > 0.0f) || !(p->temperature > 0.0f)) return fail(c, SAE_ERR_ARG, "gamma and temperature must be > 0");
    if (p->K < 0) return fail(c, SAE_ERR_ARG, "K must be >= 0");
    if ((p->learn & SAE_LEARN_TOKEN_WEIGHTS) && (p->learn & SAE_LEARN_TOKEN_EMA))
        return fail(c, SAE_ERR_ARG, "choose one token-weight rule (Algorithm 3 or the text's EMA)");
    if ((p->learn & SAE_LEARN_QUEUE_WEIGHTS) && (p->learn & SAE_LEARN_QUEUE_REL))
        return fail(c, SAE_ERR_ARG, "choose one queue-weight rule (Algorithm 2 or the text's relative rule)");
    InstState h;
    memset(&h, 0, sizeof(h));
    memcpy(h.w, p->w, sizeof(h.w));
    memcpy(h.alpha, p->alpha, sizeof(h.alpha));
    memcpy(h.mu, p->mu, sizeof(h.mu));
    memcpy(h.sigma, p->sigma, sizeof(h.sigma));
    h.gamma = p->gamma;
    h.eta = p->eta;
    h.T = p->temperature;
    h.beta = p->beta;
    h.beta_ln = p->beta_ln;
    h.K = p->K;
    h.learn = p->learn;
    const size_t nbytes = offsetof(InstState, evicted);
    int lo = inst < 0 ? 0 : inst, hi = inst < 0 ? c->dc.n_inst : inst + 1;
    for (int i = lo; i < hi; ++i) {
        hipError_t e = hipMemcpyAsync(c->dc.state + i, &h, nbytes, hipMemcpyHostToDevice, S(stream));
        if (e != hipSuccess) return hip_fail(c, e, "sae_set_params");
    }
    hipError_t e = hipStreamSynchronize(S(stream));
    if (e != hipSuccess) return hip_fail(c, e, "sae_set_params sync");
    return SAE_OK;
}

sae_status sae_get_params(sae_ctx *c, int32_t inst, sae_params *out, sae_stream_t stream)
{
    if (!c || !out) return fail(c, SAE_ERR_ARG, "ctx and out must be non-NULL");
    if (check_inst(c, inst, false) != SAE_OK) return SAE_ERR_ARG;
    InstState h;
    hipError_t e = hipMemcpyAsync(&h, c->dc.state + inst, sizeof(h), hipMemcpyDeviceToHost, S(stream));
    if (e == hipSuccess) e = hipStreamSynchronize(S(stream));
    if (e != hipSuccess) return hip_fail(c, e, "sae_get_params");
    memcpy(out->w, h.w, sizeof(out->w));
    memcpy(out->alpha, h.alpha, sizeof(out->alpha));
    memcpy(out->mu, h.mu, sizeof(out->mu));
    memcpy(out->sigma, h.sigma, sizeof(out->sigma));
    out->gamma = h.gamma;
    out->eta = h.eta;
    out->temperature = h.T;
    out->beta = h.beta;
    out->beta_ln = h.beta_ln;
    out->K = h.K;
    out->learn = h.learn;
    return SAE_OK;
}

sae_status sae_get_counters(sae_ctx *c, int32_t inst, sae_counters *out, sae_stream_t stream)
{
    if (!c || !out) return fail(c, SAE_ERR_ARG, "ctx and out must be non-NULL");
    if (check_inst(c, inst, false) != SAE_OK) return SAE_ERR_ARG;
    hipError_t e = launch_feedback(c->dc, 0, 0, S(stream));  // fold the striped counters
    InstState h;
    if (e == hipSuccess) e = hipMemcpyAsync(&h, c->dc.state + inst, sizeof(h), hipMemcpyDeviceToHost, S(stream));
    if (e == hipSuccess) e = hipStreamSynchronize(S(stream));
    if (e != hipSuccess) return hip_fail(c, e, "sae_get_counters");
    memcpy(out->evicted, h.evicted, sizeof(out->evicted));
    memcpy(out->missed, h.missed, sizeof(out->missed));
    memcpy(out->hits, h.hits, sizeof(out->hits));
    memcpy(out->evictions, h.evictions, sizeof(out->evictions));
    out->eviction_count = h.ev_count;
    out->pending = h.pending;
    out->n_updates = h.n_updates;
    memcpy(out->bin_hits, h.bin_hits, sizeof(out->bin_hits));
    memcpy(out->bin_missed, h.bin_missed, sizeof(out->bin_missed));
    memcpy(out->type_hits, h.type_hits, sizeof(out->type_hits));
    memcpy(out->type_added, h.type_added, sizeof(out->type_added));
    memcpy(out->resident, h.resident, sizeof(out->resident));
    return SAE_OK;
}

sae_status sae_set_counters(sae_ctx *c, int32_t inst, const sae_counters *in, sae_stream_t stream)
{
    if (!c || !in) return fail(c, SAE_ERR_ARG, "ctx and counters must be non-NULL");
    if (check_inst(c, inst, false) != SAE_OK) return SAE_ERR_ARG;
    hipError_t e = launch_feedback(c->dc, 0, 0, S(stream));  // fold the striped counters
    InstState h;
    if (e == hipSuccess) e = hipMemcpyAsync(&h, c->dc.state + inst, sizeof(h), hipMemcpyDeviceToHost, S(stream));
    if (e == hipSuccess) e = hipStreamSynchronize(S(stream));
    if (e != hipSuccess) return hip_fail(c, e, "sae_set_counters read");
    memcpy(h.evicted, in->evicted, sizeof(h.evicted));
    memcpy(h.missed, in->missed, sizeof(h.missed));
    memcpy(h.hits, in->hits, sizeof(h.hits));
    memcpy(h.evictions, in->evictions, sizeof(h.evictions));
    h.ev_count = in->eviction_count;
    h.pending = in->pending;
    h.n_updates = in->n_updates;
    memcpy(h.bin_hits, in->bin_hits, sizeof(h.bin_hits));
    memcpy(h.bin_missed, in->bin_missed, sizeof(h.bin_missed));
    memcpy(h.type_hits, in->type_hits, sizeof(h.type_hits));
    memcpy(h.type_added, in->type_added, sizeof(h.type_added));
    memcpy(h.resident, in->resident, sizeof(h.resident));
    e = hipMemcpyAsync(c->dc.state + inst, &h, sizeof(h), hipMemcpyHostToDevice, S(stream));
    if (e == hipSuccess) e = hipStreamSynchronize(S(stream));
    if (e != hipSuccess) return hip_fail(c, e, "sae_set_counters write");
    return SAE_OK;
}

// Blob of sae_save_state: this header, the instance's InstState (counters
// folded in), its interval buffers [Q][SAE_IVL_CAP] (when the context has a
// log-normal queue) and its recently_evicted ring [ring_cap].
struct StateHeader {
    uint32_t magic, version;
    int32_t Q, N, max_k, W, ring_cap, has_ivl;
    int32_t kind[SAE_MAX_QUEUES];
    uint64_t state_bytes, ivl_bytes, ring_bytes, total;
};
constexpr uint32_t kStateMagic = 0x53414553u;  // "SEAS"

static StateHeader state_header(const sae_ctx *c)
{
    StateHeader h;
    memset(&h, 0, sizeof(h));
    const DevCtx &d = c->dc;
    h.magic = kStateMagic;
    h.version = 1;
    h.Q = d.Q;
    h.N = d.N;
    h.max_k = d.max_k;
    h.W = d.W;
    h.ring_cap = d.ring_cap;
    h.has_ivl = d.ln_mask ? 1 : 0;
    for (int q = 0; q < SAE_MAX_QUEUES; ++q) h.kind[q] = q < d.Q ? d.kind[q] : -1;
    h.state_bytes = sizeof(InstState);
    h.ivl_bytes = h.has_ivl ? (uint64_t)d.Q * SAE_IVL_CAP * sizeof(int32_t) : 0;
    h.ring_bytes = (uint64_t)d.ring_cap * sizeof(GhostEntry);
    h.total = sizeof(StateHeader) + h.state_bytes + h.ivl_bytes + h.ring_bytes;
    return h;
}

sae_status sae_state_size(sae_ctx *c, size_t *bytes)
{
    if (!c || !bytes) return fail(c, SAE_ERR_ARG, "ctx and bytes must be non-NULL");
    *bytes = (size_t)state_header(c).total;
    return SAE_OK;
}

sae_status sae_save_state(sae_ctx *c, int32_t inst, void *buf, size_t bytes, sae_stream_t stream)
{
    if (!c || !buf) return fail(c, SAE_ERR_ARG, "ctx and buf must be non-NULL");
    if (check_inst(c, inst, false) != SAE_OK) return SAE_ERR_ARG;
    const StateHeader h = state_header(c);
    if (bytes != h.total) return fail(c, SAE_ERR_ARG, "bytes must be sae_state_size()");
    char *p = static_cast<char *>(buf);
    memcpy(p, &h, sizeof(h));
    const DevCtx &d = c->dc;
    hipError_t e = launch_feedback(d, 0, 0, S(stream));  // fold the striped counters
    if (e == hipSuccess)
        e = hipMemcpyAsync(p + sizeof(h), d.state + inst, h.state_bytes, hipMemcpyDeviceToHost, S(stream));
    if (e == hipSuccess && h.ivl_bytes)
        e = hipMemcpyAsync(p + sizeof(h) + h.state_bytes, d.ivl + (long long)inst * d.Q * SAE_IVL_CAP, h.ivl_bytes,
                           hipMemcpyDeviceToHost, S(stream));
    if (e == hipSuccess)
        e = hipMemcpyAsync(p + sizeof(h) + h.state_bytes + h.ivl_bytes, d.ring + (long long)inst * d.ring_cap,
                           h.ring_bytes, hipMemcpyDeviceToHost, S(stream));
    if (e == hipSuccess) e = hipStreamSynchronize(S(stream));
    if (e != hipSuccess) return hip_fail(c, e, "sae_save_state");
    return SAE_OK;
}

sae_status sae_load_state(sae_ctx *c, int32_t inst, const void *buf, size_t bytes, sae_stream_t stream)
{
    if (!c || !buf) return fail(c, SAE_ERR_ARG, "ctx and buf must be non-NULL");
    if (check_inst(c, inst, false) != SAE_OK) return SAE_ERR_ARG;
    const StateHeader h = state_header(c);
    StateHeader got;
    if (bytes < sizeof(got)) return fail(c, SAE_ERR_ARG, "blob too small");
    memcpy(&got, buf, sizeof(got));
    if (bytes != h.total || memcmp(&got, &h, sizeof(h)) != 0)
        return fail(c, SAE_ERR_ARG, "blob of another context shape, version or size");
    const char *p = static_cast<const char *>(buf);
    const DevCtx &d = c->dc;
    // fold (and so empty) the striped counters first: the blob's totals replace them
    hipError_t e = launch_feedback(d, 0, 0, S(stream));
    if (e == hipSuccess)
        e = hipMemcpyAsync(d.state + inst, p + sizeof(h), h.state_bytes, hipMemcpyHostToDevice, S(stream));
    if (e == hipSuccess && h.ivl_bytes)
        e = hipMemcpyAsync(d.ivl + (long long)inst * d.Q * SAE_IVL_CAP, p + sizeof(h) + h.state_bytes, h.ivl_bytes,
                           hipMemcpyHostToDevice, S(stream));
    if (e == hipSuccess)
        e = hipMemcpyAsync(d.ring + (long long)inst * d.ring_cap, p + sizeof(h) + h.state_bytes + h.ivl_bytes,
                           h.ring_bytes, hipMemcpyHostToDevice, S(stream));
    if (e == hipSuccess) e = launch_ghost_rebuild(d, S(stream));
    if (e == hipSuccess) e = hipStreamSynchronize(S(stream));
    if (e != hipSuccess) return hip_fail(c, e, "sae_load_state");
    c->ghost_tombs = 0;
    return SAE_OK;
}

sae_status sae_get_intervals(sae_ctx *c, int32_t inst, int32_t queue, int32_t *out, int32_t cap, int32_t *n,
                             sae_stream_t stream)
{
    if (!c || !n || cap < 0 || (cap > 0 && !out)) return fail(c, SAE_ERR_ARG, "ctx, n (and out if cap > 0) needed");
    if (check_inst(c, inst, false) != SAE_OK) return SAE_ERR_ARG;
    if (queue < 0 || queue >= c->dc.Q || c->dc.kind[queue] != SAE_KIND_LOGNORMAL)
        return fail(c, SAE_ERR_ARG, "queue is not a log-normal queue");
    InstState h;
    hipError_t e = hipMemcpyAsync(&h, c->dc.state + inst, sizeof(h), hipMemcpyDeviceToHost, S(stream));
    if (e == hipSuccess) e = hipStreamSynchronize(S(stream));
    if (e != hipSuccess) return hip_fail(c, e, "sae_get_intervals");
    const long long total = h.ivl_n[queue];
    long long lo = total - SAE_IVL_CAP;
    if (lo < h.ivl_start[queue]) lo = h.ivl_start[queue];
    const long long cnt = total - lo;
    *n = (int32_t)cnt;
    const long long want = cnt < cap ? cnt : cap;
    const int32_t *ring = c->dc.ivl + ((long long)inst * c->dc.Q + queue) * SAE_IVL_CAP;
    for (long long done = 0; done < want && e == hipSuccess;) {
        const long long pos = (lo + done) % SAE_IVL_CAP;
        long long len = SAE_IVL_CAP - pos;
        if (len > want - done) len = want - done;
        e = hipMemcpyAsync(out + done, ring + pos, (size_t)len * sizeof(int32_t), hipMemcpyDeviceToHost, S(stream));
        done += len;
    }
    if (e == hipSuccess) e = hipStreamSynchronize(S(stream));
    if (e != hipSuccess) return hip_fail(c, e, "sae_get_intervals copy");
    return SAE_OK;
}

// Argument checks shared by both predictor entry points (work may be NULL for
// the one that brings its own buffer).
static sae_status predict_args(int32_t n, int32_t d, const uint16_t *h, const sae_predictor *w, const float *work,
                               bool need_work, const float *logit)
{
    if (n < 0) return fail(nullptr, SAE_ERR_ARG, "n must be >= 0");
    if (d < 256 || d > 16384 || d % 256 != 0)
        return fail(nullptr, SAE_ERR_ARG, "d must be a multiple of 256 in 256..16384");
    if (n == 0) return SAE_OK;
    if (!h || !w || !w->w1 || !w->b1 || !w->w2 || !w->b2 || !w->w3 || !w->b3 || (need_work && !work) || !logit)
        return fail(nullptr, SAE_ERR_ARG, "h, every weight, work and logit must be non-NULL");
    if (!aligned(h, 16) || !aligned(w->w1, 16) || !aligned(w->w2, 16) || (need_work && !aligned(work, 16)))
        return fail(nullptr, SAE_ERR_ARG, "h, w1, w2 and work must be 16-byte aligned");
    return SAE_OK;
}

sae_status sae_predict_sessions(int32_t n, int32_t d, const uint16_t *h, const sae_predictor *w, float *work,
                                float *logit, uint8_t *pred, sae_stream_t stream)
{
    sae_status st = predict_args(n, d, h, w, work, true, logit);
    if (st != SAE_OK || n == 0) return st;
    hipError_t e = launch_predict(n, d, h, w->w1, w->b1, w->w2, w->b2, w->w3, w->b3, work, logit, pred, S(stream));
    if (e != hipSuccess) return hip_fail(nullptr, e, "sae_predict_sessions");
    return SAE_OK;
}

sae_status sae_predict_sessions_noalloc(int32_t n, int32_t d, const uint16_t *h, const sae_predictor *w,
                                        float *logit, uint8_t *pred, sae_stream_t stream)
{
    if (n > SAE_PRED_NOALLOC_MAX_N)
        return fail(nullptr, SAE_ERR_ARG, "n exceeds SAE_PRED_NOALLOC_MAX_N (4096) rows");
    sae_status st = predict_args(n, d, h, w, nullptr, false, logit);
    if (st != SAE_OK || n == 0) return st;
    float *work = nullptr;
    hipError_t e = predict_scratch(&work);
    if (e != hipSuccess) return hip_fail(nullptr, e, "sae_predict_sessions_noalloc: library buffer");
    e = launch_predict(n, d, h, w->w1, w->b1, w->w2, w->b2, w->w3, w->b3, work, logit, pred, S(stream));
    if (e != hipSuccess) return hip_fail(nullptr, e, "sae_predict_sessions_noalloc");
    return SAE_OK;
}

sae_status sae_block_type(const uint8_t *counts, int64_t n, uint8_t *tau, sae_stream_t stream)
{
    if (n < 0 || (n > 0 && (!counts || !tau))) return fail(nullptr, SAE_ERR_ARG, "counts/tau must be non-NULL, n >= 0");
    hipError_t e = launch_block_type(counts, n, tau, S(stream));
    if (e != hipSuccess) return hip_fail(nullptr, e, "sae_block_type");
    return SAE_OK;
}

sae_status sae_recipe_eval(int32_t fn, int64_t n, const float *x, float *y, sae_stream_t stream)
{
    if (fn != SAE_FN_LN && fn != SAE_FN_EXP && fn != SAE_FN_ERFC) return fail(nullptr, SAE_ERR_ARG, "unknown recipe function");
    if (n < 0 || (n > 0 && (!x || !y))) return fail(nullptr, SAE_ERR_ARG, "x/y must be non-NULL, n >= 0");
    hipError_t e = launch_recipe_eval(fn, n, x, y, S(stream));
    if (e != hipSuccess) return hip_fail(nullptr, e, "sae_recipe_eval");
    return SAE_OK;
}

sae_status sae_classify_blocks(sae_ctx *c, int32_t n, const uint8_t *hint, uint16_t *meta, const int32_t *roles,
                               sae_stream_t stream)
{
    if (!c) return fail(c, SAE_ERR_ARG, "ctx must be non-NULL");
    if (n < 0) return fail(c, SAE_ERR_ARG, "n must be >= 0");
    if (n == 0) return SAE_OK;
    if (!hint || !meta || !roles) return fail(c, SAE_ERR_ARG, "hint, meta, roles must be non-NULL");
    for (int r = 0; r < SAE_N_ROLES; ++r)
        if (roles[r] < 0 || roles[r] >= c->cfg.n_queues)
            return fail(c, SAE_ERR_ARG, "roles[] must be queue indices below n_queues");
    hipError_t e = launch_classify(n, hint, meta, roles, S(stream));
    if (e != hipSuccess) return hip_fail(c, e, "sae_classify_blocks");
    return SAE_OK;
}

sae_status sae_index_build(sae_ctx *c, sae_stream_t stream)
{
    if (!c) return fail(c, SAE_ERR_ARG, "ctx must be non-NULL");
    if (!c->pool_bound) return fail(c, SAE_ERR_STATE, "no pool bound");
    hipError_t e = launch_index_build(c->dc, S(stream));
    if (e != hipSuccess) return hip_fail(c, e, "sae_index_build");
    c->index_tombs = 0;
    c->ghost_tombs = 0;
    return SAE_OK;
}

sae_status sae_insert_blocks(sae_ctx *c, int32_t n, const int32_t *inst, const int32_t *ids, const uint64_t *hash,
                             const int32_t *parent, const int32_t *last_access, const uint16_t *meta,
                             const uint32_t *off, sae_stream_t stream)
{
    if (!c) return fail(c, SAE_ERR_ARG, "ctx must be non-NULL");
    if (!c->pool_bound) return fail(c, SAE_ERR_STATE, "no pool bound");
    if (n < 0 || n > c->skip_cap) return fail(c, SAE_ERR_ARG, "n must be in 0..n_instances*blocks_per_instance");
    if (n == 0) return SAE_OK;
    if (!ids || !hash || !parent || !last_access || !meta || !off)
        return fail(c, SAE_ERR_ARG, "ids, hash, parent, last_access, meta, off must be non-NULL");
    hipError_t e = launch_insert(c->dc, n, inst, ids, hash, parent, last_access, meta, off, c->skip, S(stream));
    if (e != hipSuccess) return hip_fail(c, e, "sae_insert_blocks");
    c->ghost_tombs += n;
    if (c->ghost_tombs > 0.25 * (double)c->ghost_slots) {
        e = launch_ghost_rebuild(c->dc, S(stream));
        if (e != hipSuccess) return hip_fail(c, e, "ghost rebuild");
        c->ghost_tombs = 0;
    }
    return SAE_OK;
}

sae_status sae_ref_blocks(sae_ctx *c, int32_t n, const int32_t *inst, const int32_t *ids, int32_t delta,
                          sae_stream_t stream)
{
    if (!c) return fail(c, SAE_ERR_ARG, "ctx must be non-NULL");
    if (!c->pool_bound) return fail(c, SAE_ERR_STATE, "no pool bound");
    if (n < 0) return fail(c, SAE_ERR_ARG, "n must be >= 0");
    if (n == 0) return SAE_OK;
    if (!ids) return fail(c, SAE_ERR_ARG, "ids must be non-NULL");
    hipError_t e = launch_ref(c->dc, n, inst, ids, delta, S(stream));
    if (e != hipSuccess) return hip_fail(c, e, "sae_ref_blocks");
    return SAE_OK;
}

namespace {

sae_status pm_check(sae_ctx *c, int32_t n_req, int32_t max_len, const uint64_t *hashes, const int32_t *lens,
                    uint32_t flags, int32_t *match_len, int32_t *matched_ids)
{
    if (!c) return fail(c, SAE_ERR_ARG, "ctx must be non-NULL");
    if (!c->pool_bound) return fail(c, SAE_ERR_STATE, "no pool bound");
    if (n_req < 0 || max_len < 0) return fail(c, SAE_ERR_ARG, "n_req and max_len must be >= 0");
    if (flags & ~(uint32_t)(SAE_PM_TOUCH | SAE_PM_STATS | SAE_PM_INTERVALS))
        return fail(c, SAE_ERR_ARG, "unknown prefix-match flag");
    if (n_req == 0) return SAE_OK;
    if (max_len < 1 || !hashes || !lens || !match_len)
        return fail(c, SAE_ERR_ARG, "hashes, lens, match_len must be non-NULL and max_len >= 1");
    if (flags & SAE_PM_INTERVALS) {
        if (!matched_ids) return fail(c, SAE_ERR_ARG, "SAE_PM_INTERVALS needs matched_ids");
        if (n_req > c->dc.max_req) return fail(c, SAE_ERR_ARG, "SAE_PM_INTERVALS: n_req exceeds max_requests");
    }
    if ((long long)n_req * SAE_WAVE > 0x7FFFFFFFll) return fail(c, SAE_ERR_ARG, "n_req too large");
    return SAE_OK;
}

}  // namespace

sae_status sae_prefix_match(sae_ctx *c, int32_t n_req, int32_t max_len, const uint64_t *hashes, const int32_t *lens,
                            const int32_t *inst, int32_t now, uint32_t flags, int32_t *match_len,
                            int32_t *matched_ids, sae_stream_t stream)
{
    const sae_status st = pm_check(c, n_req, max_len, hashes, lens, flags, match_len, matched_ids);
    if (st != SAE_OK || n_req == 0) return st;
    hipError_t e = launch_prefix_match(c->dc, n_req, max_len, hashes, lens, inst, now, flags, match_len,
                                       matched_ids, S(stream));
    if (e != hipSuccess) return hip_fail(c, e, "sae_prefix_match");
    return SAE_OK;
}

namespace {

sae_status ss_check(sae_ctx *c, int32_t now, int32_t k, const int32_t *k_per_inst, uint32_t flags, int32_t *victims,
                    float *scores, int32_t *count, int32_t *decision, int32_t *decision_count, SelectArgs &a,
                    bool &batched)
{
    if (!c) return fail(c, SAE_ERR_ARG, "ctx must be non-NULL");
    if (!c->pool_bound) return fail(c, SAE_ERR_STATE, "no pool bound");
    const uint32_t known =
        SAE_SS_COMMIT | SAE_SS_ENGINE_SCAN | SAE_SS_ENGINE_BATCHED | SAE_SS_FORCE_FALLBACK | SAE_SS_CASCADE;
    if (flags & ~known) return fail(c, SAE_ERR_ARG, "unknown score-select flag");
    if ((flags & SAE_SS_CASCADE) && c->dc.max_k > 4096)
        return fail(c, SAE_ERR_ARG, "SAE_SS_CASCADE needs max_k <= 4096");
    if ((flags & SAE_SS_ENGINE_SCAN) && (flags & SAE_SS_ENGINE_BATCHED))
        return fail(c, SAE_ERR_ARG, "choose at most one engine");
    if (!k_per_inst && (k < 0 || k > c->dc.max_k)) return fail(c, SAE_ERR_ARG, "k must be in 0..max_k");
    if (!victims || !count || !decision || !decision_count)
        return fail(c, SAE_ERR_ARG, "victims, count, decision, decision_count must be non-NULL");
    if (flags & SAE_SS_ENGINE_BATCHED) {
        if (!batched_engine_fits(c->dc))
            return fail(c, SAE_ERR_ARG, "batched engine needs <= 65536 blocks per instance and Q*max_k to fit LDS");
        batched = true;
    } else if (flags & (SAE_SS_ENGINE_SCAN | SAE_SS_FORCE_FALLBACK)) {
        batched = false;
    } else {
        batched = batched_engine_fits(c->dc) && (c->dc.n_inst >= 32 || c->dc.N <= 16384);
    }
    a.now = now;
    a.k = k;
    a.k_per_inst = k_per_inst;
    a.flags = flags;
    a.victims = victims;
    a.scores = scores;
    a.count = count;
    a.decision = decision;
    a.decision_count = decision_count;
    return SAE_OK;
}

// The selection's launches; with pm (pool-scan engine only), the prefix match
// pm shares the launch of the selection's sampling and bounds.
sae_status ss_run(sae_ctx *c, const SelectArgs &a, bool batched, hipStream_t s, const PmArgs *pm)
{
    const uint32_t flags = a.flags;
    hipError_t e;
    if (batched) {
        e = launch_select_batched(c->dc, a, s);
    } else {
        hipEvent_t e0 = nullptr, e1 = nullptr;
        if (c->prof) {
            if (c->prof_free.empty()) {
                hipEvent_t x, y;
                if (hipEventCreate(&x) != hipSuccess || hipEventCreate(&y) != hipSuccess)
                    return fail(c, SAE_ERR_HIP, "hipEventCreate");
                c->prof_free.push_back({x, y});
            }
            auto pr = c->prof_free.back();
            c->prof_free.pop_back();
            c->prof_used.push_back(pr);
            e0 = pr.first;
            e1 = pr.second;
        }
        e = launch_select_scan(c->dc, a, s, e0, e1, pm, &c->prep_calls);
    }
    if (e == hipSuccess && (flags & SAE_SS_CASCADE)) {
        e = launch_cascade(c->dc, a, s, c->casc_set);
        c->casc_set ^= 1;
    }
    if (e != hipSuccess) return hip_fail(c, e, pm ? "sae_match_select" : "sae_score_select");
    if (flags & SAE_SS_COMMIT) {
        e = launch_commit(c->dc, a, s);
        if (e != hipSuccess) return hip_fail(c, e, "commit");
        double d = (double)c->dc.max_k;
        c->index_tombs += d;
        c->ghost_tombs += d;
        if (c->index_tombs > 0.25 * (double)(c->index_slots - c->dc.N)) {
            e = launch_index_rebuild(c->dc, s);
            if (e != hipSuccess) return hip_fail(c, e, "index rebuild");
            c->index_tombs = 0;
        }
        if (c->ghost_tombs > 0.25 * (double)c->ghost_slots) {
            e = launch_ghost_rebuild(c->dc, s);
            if (e != hipSuccess) return hip_fail(c, e, "ghost rebuild");
            c->ghost_tombs = 0;
        }
    }
    return SAE_OK;
}

}  // namespace

sae_status sae_score_select(sae_ctx *c, int32_t now, int32_t k, const int32_t *k_per_inst, uint32_t flags,
                            int32_t *victims, float *scores, int32_t *count, int32_t *decision,
                            int32_t *decision_count, sae_stream_t stream)
{
    SelectArgs a;
    bool batched = false;
    const sae_status st =
        ss_check(c, now, k, k_per_inst, flags, victims, scores, count, decision, decision_count, a, batched);
    if (st != SAE_OK) return st;
    return ss_run(c, a, batched, S(stream), nullptr);
}

sae_status sae_match_select(sae_ctx *c, int32_t n_req, int32_t max_len, const uint64_t *hashes, const int32_t *lens,
                            const int32_t *inst, int32_t pm_now, uint32_t pm_flags, int32_t *match_len,
                            int32_t *matched_ids, int32_t now, int32_t k, const int32_t *k_per_inst,
                            uint32_t flags, int32_t *victims, float *scores, int32_t *count, int32_t *decision,
                            int32_t *decision_count, sae_stream_t stream)
{
    sae_status st = pm_check(c, n_req, max_len, hashes, lens, pm_flags, match_len, matched_ids);
    if (st != SAE_OK) return st;
    SelectArgs a;
    bool batched = false;
    st = ss_check(c, now, k, k_per_inst, flags, victims, scores, count, decision, decision_count, a, batched);
    if (st != SAE_OK) return st;
    hipStream_t s = S(stream);
    if (batched || n_req == 0) {
        // the batched engine has no separate sampling step: the two calls in turn
        if (n_req > 0) {
            hipError_t e = launch_prefix_match(c->dc, n_req, max_len, hashes, lens, inst, pm_now, pm_flags, match_len,
                                               matched_ids, s);
            if (e != hipSuccess) return hip_fail(c, e, "sae_match_select");
        }
        return ss_run(c, a, batched, s, nullptr);
    }
    const PmArgs pm = {n_req, max_len, hashes, lens, inst, pm_now, pm_flags, match_len, matched_ids};
    return ss_run(c, a, false, s, &pm);
}

sae_status sae_feedback_update(sae_ctx *c, uint32_t flags, sae_stream_t stream)
{
    if (!c) return fail(c, SAE_ERR_ARG, "ctx must be non-NULL");
    if (flags & ~(uint32_t)SAE_FB_FORCE) return fail(c, SAE_ERR_ARG, "unknown feedback flag");
    hipError_t e = launch_feedback(c->dc, flags, 1, S(stream));
    if (e != hipSuccess) return hip_fail(c, e, "sae_feedback_update");
    return SAE_OK;
}

sae_status sae_poll_status(sae_ctx *c, sae_stream_t stream, uint32_t *bits)
{
    if (!c || !bits) return fail(c, SAE_ERR_ARG, "ctx and bits must be non-NULL");
    uint32_t h = 0;
    hipError_t e = hipMemcpyAsync(&h, c->dc.status, sizeof(h), hipMemcpyDeviceToHost, S(stream));
    if (e == hipSuccess) e = hipStreamSynchronize(S(stream));
    if (e == hipSuccess) e = hipMemsetAsync(c->dc.status, 0, sizeof(uint32_t), S(stream));
    if (e == hipSuccess) e = hipStreamSynchronize(S(stream));
    if (e != hipSuccess) return hip_fail(c, e, "sae_poll_status");
    *bits = h;
    return SAE_OK;
}

sae_status sae_select_stats(sae_ctx *c, int32_t inst, uint32_t *out, sae_stream_t stream)
{
    if (!c || !out) return fail(c, SAE_ERR_ARG, "ctx and out must be non-NULL");
    if (check_inst(c, inst, false) != SAE_OK) return SAE_ERR_ARG;
    hipError_t e = hipMemcpyAsync(out, c->dc.sel_stats + (long long)inst * c->dc.Q * 4, sizeof(uint32_t) * 4 * c->dc.Q,
                                  hipMemcpyDeviceToHost, S(stream));
    if (e == hipSuccess) e = hipStreamSynchronize(S(stream));
    if (e != hipSuccess) return hip_fail(c, e, "sae_select_stats");
    return SAE_OK;
}

sae_status sae_profile_enable(sae_ctx *c, int32_t enable)
{
    if (!c) return fail(c, SAE_ERR_ARG, "ctx must be non-NULL");
    c->prof = enable != 0;
    return SAE_OK;
}

sae_status sae_profile_read(sae_ctx *c, double *ms, int64_t *launches)
{
    if (!c || !ms || !launches) return fail(c, SAE_ERR_ARG, "ctx, ms, launches must be non-NULL");
    double tot = 0;
    int64_t n = 0;
    for (auto &p : c->prof_used) {
        hipError_t e = hipEventSynchronize(p.second);
        if (e != hipSuccess) return hip_fail(c, e, "sae_profile_read");
        float t = 0;
        e = hipEventElapsedTime(&t, p.first, p.second);
        if (e != hipSuccess) return hip_fail(c, e, "sae_profile_read");
        tot += t;
        ++n;
        c->prof_free.push_back(p);
    }
    c->prof_used.clear();
    *ms = tot;
    *launches = n;
    return SAE_OK;
}

}  // extern "C"
