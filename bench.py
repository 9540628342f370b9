"""Benchmark of the eviction hot path on one MI355X.

Workload (the large-pool configuration): one cache of 4,194,304 blocks (64M
tokens), 5 queues (evict-first, structural, chat log-normal, agent
log-normal, recency), k = 4,096 victims per queue, and a batch of 4,096
prefix-match requests of 128 block hashes.

A step is one full pass of the hot path on one cache:
  sae_match_select: the prefix match (touch + stats), then the selection
  (every block scored, per-queue k smallest, Algorithm 1 decision, commit),
  the selection's sampling and bounds running in the prefix match's launch
  -> sae_feedback_update.
Steps rotate over R independent caches (own pool, index and recently-evicted
table) so that the working set exceeds the 256 MB last-level cache and the
pool is read from HBM.

value = blocks scored+selected per second over the timed steps (G blk/s).
The JSON line also carries:
  * roofline: the score+select pass (bytes the scoring must read / the pass's
    HIP-event-timed duration), with the scan kernel's own figure inside;
  * the score+select call alone, alone beside a read-only prefix match on a
    second stream, with a cascading decision, with every learner on;
  * step_two_calls: the same step with sae_prefix_match and sae_score_select
    as two calls;
  * steady_state: the step over enough steps that the index and
    recently-evicted tables are rebuilt as in a long run; step_steady_pools:
    the step alone on the pools that leg left (decisions mostly from
    Algorithm 1's second stage);
  * configs: the other configurations' per-operation GPU times beside the
    oracle's host time (tiny pool, mid pool, trace replay, batched sweep),
    and the batched sweep's fixed-against-learned comparison over its full
    10,000 requests per cache (two child processes);
  * cpu_baseline: the oracle on a bounded sample of the same workload.
"""
import argparse
import hashlib
import json
import os
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "cached blocks scored+selected per sec (G blk/s) at 4M blocks; % HBM peak"
HBM_PEAK_GBS = 8000.0
BYTES_PER_BLOCK = 10  # last_access 4 + meta 2 + off 4: what the scoring pass must read
PASS_KERNEL_SOURCES = ["paper_2605_18825_amd/csrc/k_select.hip", "paper_2605_18825_amd/csrc/sae_internal.h",
                       "paper_2605_18825_amd/csrc/pm_match.h"]


def kernel_source_hash():
    h = hashlib.sha256()
    for f in PASS_KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(name="score_select_large_pool_traffic.json"):
    """HBM bytes per launch of a pass's kernels from rocprofv3 counters, if
    the committed measurement was taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    return t


def note(msg):
    """Progress on stderr (the JSON line is the only stdout output)."""
    print("bench: " + msg, file=sys.stderr, flush=True)


def cores():
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# ---------------------------------------------------------------------------- CPU legs
def oracle_cache(cfg, pool):
    import oracle
    prm = oracle.Params(len(cfg["kinds"]), mu=cfg["mu"], sigma=cfg["sigma"], K=cfg["k"])
    oc = oracle.OracleCache(pool["n_blocks"], cfg["kinds"], prm)
    oc.bind(pool["last_access"], pool["queue"], oracle.block_type(pool["counts"]), pool["ntok"], pool["ob"],
            pool["omax"], pool["valid"], pool["ref_count"], pool["parent"], pool["hash"], pool.get("access_count"))
    return oc


def cpu_baseline(cfg, pool, reqs, lens, budget_s):
    """The oracle as it stands, single-threaded on the host, on a bounded number
    of full steps of the same workload."""
    oc = oracle_cache(cfg, pool)
    now = pool["now"]
    steps, t0 = 0, time.perf_counter()
    while True:
        oc.prefix_match(reqs, lens, now, touch=True, stats=True)
        oc.score_select(now, cfg["k"], commit=True)
        oc.feedback()
        steps += 1
        now += 1000
        el = time.perf_counter() - t0
        if el >= budget_s or steps >= 50:
            break
    return dict(value=pool["n_blocks"] * steps / el / 1e9, unit="G blk/s", cores=1, kind="oracle",
                sample="%d full step(s) (prefix match of 4096x128 hashes, score+select+commit of 4,194,304 "
                       "blocks, feedback) on one host core, %.1f s" % (steps, el))


def cpu_recency_lists(cfg, pool, reps=10):
    """A faster exact CPU selection (per-(queue, type) recency lists, the
    per-queue heap idea) on the same pool: score+select without commit, timed
    apart from building the lists (which a live cache keeps up incrementally);
    the oracle's full-sort selection of the same call is timed beside it and
    the two decisions are compared."""
    import numpy as np
    from oracle.recency import RecencyLists
    oc = oracle_cache(cfg, pool)
    now, k = pool["now"], cfg["k"]
    t0 = time.perf_counter()
    rl = RecencyLists(oc)
    t_build = time.perf_counter() - t0
    t0 = time.perf_counter()
    for _ in range(reps):
        _, _, dec = rl.score_select(now, k)
    t_sel = (time.perf_counter() - t0) / reps
    t0 = time.perf_counter()
    _, _, dec_o = oc.score_select(now, k)
    t_or = time.perf_counter() - t0
    return dict(value=pool["n_blocks"] / t_sel / 1e9, unit="G blk/s", cores=1, kind="recency lists (exact)",
                ms_per_select=t_sel * 1e3, build_s=t_build, blocks_scored=int(rl.visited),
                oracle_select_ms=t_or * 1e3, same_decision_as_oracle=bool(np.array_equal(dec, dec_o)),
                sample="%d score+select calls (no commit) on one host core; log-normal and recency queues walk "
                       "their per-type lists, the structural queue is scanned whole" % reps)


def _oracle_select_instance(job):
    """One batched-sweep cache's score+select on the oracle (a worker process)."""
    cfg, seed, k = job
    import synth
    pool = synth.make_pool(cfg, seed=seed)
    oc = oracle_cache(cfg, pool)
    t0 = time.perf_counter()
    oc.score_select(pool["now"], k)
    return time.perf_counter() - t0


# ---------------------------------------------------------------------------- GPU helpers
class Timer:
    """HIP events on one stream around a loop of calls."""

    def __init__(self, stream):
        import torch
        self.stream = stream
        self.a = torch.cuda.Event(enable_timing=True)
        self.b = torch.cuda.Event(enable_timing=True)

    def __enter__(self):
        self.a.record(self.stream)
        return self

    def __exit__(self, *exc):
        import torch
        self.b.record(self.stream)
        torch.cuda.synchronize()
        self.ms = self.a.elapsed_time(self.b)


def make_cache(api, DevicePool, SelectBuffers, cfg, pool, n_inst=1, max_requests=0, learn=3):
    N, Q, k = pool["n_blocks"], len(cfg["kinds"]), cfg["k"]
    ctx = api.sae_create(n_inst, N, cfg["kinds"], max_k=cfg.get("max_k", k), max_requests=max_requests)
    dp = DevicePool(n_inst, N)
    for i in range(n_inst):
        dp.fill_instance(i, pool)
    dp.bind(ctx)
    api.sae_index_build(ctx)
    api.sae_set_params(ctx, -1, api.make_params(Q, mu=cfg["mu"], sigma=cfg["sigma"], K=k, learn=learn))
    return dict(ctx=ctx, dp=dp, out=SelectBuffers(n_inst, Q, cfg.get("max_k", k)), now=pool["now"])


# ---------------------------------------------------------------------------- config legs
def leg_tiny(api, DevicePool, SelectBuffers, stream, with_cpu):
    """Tiny pool: 4,096 blocks, 3 queues, k = 64; 256 requests of up to 32 hashes."""
    import numpy as np
    import torch
    import synth
    cfg = synth.pool_config("tiny")
    pool = synth.make_pool(cfg)
    reqs, lens = synth.make_requests(pool["chains"], cfg["n_req"], cfg["req_len"], cfg["hit_frac"], cfg["seed"] + 1)
    c = make_cache(api, DevicePool, SelectBuffers, cfg, pool)
    hd = torch.as_tensor(np.asarray(reqs, np.uint64).view(np.int64)).cuda()
    ld = torch.as_tensor(lens).cuda()
    ml = torch.zeros(len(lens), dtype=torch.int32, device="cuda")
    reps = 200
    with torch.cuda.stream(stream):
        for _ in range(10):
            c["out"].run(c["ctx"], c["now"], cfg["k"], 0, stream=stream)
        with Timer(stream) as ts:
            for _ in range(reps):
                c["out"].run(c["ctx"], c["now"], cfg["k"], 0, stream=stream)
        with Timer(stream) as tp:
            for i in range(reps):
                api.sae_prefix_match(c["ctx"], hd, ld, c["now"] + i, api.PM_TOUCH | api.PM_STATS, ml, stream=stream)
    api.sae_destroy(c["ctx"])
    res = dict(workload="4,096 blocks, 3 queues, k=64; 256 requests x up to 32 hashes",
               gpu_score_select_us=ts.ms * 1e3 / reps, gpu_prefix_match_us=tp.ms * 1e3 / reps)
    if with_cpu:
        oc = oracle_cache(cfg, pool)
        n, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < 1.0:
            oc.score_select(pool["now"], cfg["k"])
            n += 1
        res["cpu_score_select_us"] = (time.perf_counter() - t0) * 1e6 / n
        n, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < 1.0:
            oc.prefix_match(reqs, lens, pool["now"] + n, touch=True, stats=True)
            n += 1
        res["cpu_prefix_match_us"] = (time.perf_counter() - t0) * 1e6 / n
        res["cpu_cores"] = 1
    return res


def leg_mid(api, DevicePool, SelectBuffers, stream, with_cpu):
    """Mid pool: 262,144 blocks, 3 queues, k = 1,024: a decision (score,
    select, commit) and the feedback update, 64 times in a row."""
    import torch
    import synth
    cfg = synth.pool_config("mid")
    pool = synth.make_pool(cfg)
    c = make_cache(api, DevicePool, SelectBuffers, cfg, pool)
    nd = cfg["n_decisions"]
    with torch.cuda.stream(stream):
        with Timer(stream) as t:
            now = c["now"]
            for _ in range(nd):
                c["out"].run(c["ctx"], now, cfg["k"], api.SS_COMMIT, stream=stream)
                api.sae_feedback_update(c["ctx"], 0, stream=stream)
                now += 1000
    api.sae_destroy(c["ctx"])
    res = dict(workload="262,144 blocks, 3 queues, k=1024; %d decisions with commit and feedback" % nd,
               gpu_decision_us=t.ms * 1e3 / nd, gpu_blocks_per_s=pool["n_blocks"] * nd / (t.ms * 1e-3))
    if with_cpu:
        oc = oracle_cache(cfg, pool)
        now, n, t0 = pool["now"], 0, time.perf_counter()
        while n < 4:
            oc.score_select(now, cfg["k"], commit=True)
            oc.feedback()
            now += 1000
            n += 1
        el = time.perf_counter() - t0
        res.update(cpu_decision_us=el * 1e6 / n, cpu_blocks_per_s=pool["n_blocks"] * n / el, cpu_cores=1,
                   cpu_sample="%d decisions" % n)
    return res


def leg_trace(stream, with_cpu):
    """Trace replay, balanced mix, one 36K-token cache with Algorithms 2 and 3:
    requests per second of the whole replay (the host-side block manager, the
    C-ABI calls and their read-backs), GPU against the oracle."""
    import torch
    from paper_2605_18825_amd.engine import DeviceBackend
    from synth.replay import Replay
    from synth.trace import TRACE_CONFIGS, TRACE_KINDS, TRACE_MU, TRACE_ROLES, TRACE_SIGMA, trace_gen
    cfg = TRACE_CONFIGS["trace_balanced"]
    warm, steps = 500, 2000
    gen = trace_gen("trace_balanced", 0)
    reqs = [gen.next() for _ in range(warm + steps)]
    dev = DeviceBackend(1, cfg["capacity"], TRACE_KINDS, TRACE_ROLES, cfg["max_k"], TRACE_MU, TRACE_SIGMA, cfg["K"], 3)
    rep = Replay(dev, 1, cfg["capacity"], cfg["k_min"], cfg["max_k"], cfg["concurrency"])
    with torch.cuda.stream(dev.stream):
        for r in reqs[:warm]:
            rep.step({0: r})
        torch.cuda.synchronize()
        d0 = rep.summary()["decisions"]
        t0 = time.perf_counter()
        for r in reqs[warm:]:
            rep.step({0: r})
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
    dec = rep.summary()["decisions"] - d0
    dev.close()
    res = dict(workload="balanced trace, 2,250-block cache, Algorithms 2/3; %d requests after %d" % (steps, warm),
               gpu_requests_per_s=steps / el, gpu_decisions_per_request=dec / steps,
               gpu_note="end to end: host block manager, C-ABI calls and read-backs per request")
    if with_cpu:
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        from oracle_backend import OracleBackend
        orc = OracleBackend([0], cfg["capacity"], TRACE_KINDS, TRACE_ROLES, TRACE_MU, TRACE_SIGMA, cfg["K"], 3)
        ro = Replay(orc, 1, cfg["capacity"], cfg["k_min"], cfg["max_k"], cfg["concurrency"], insts=[0])
        for r in reqs[:warm]:
            ro.step({0: r})
        n, t0 = 0, time.perf_counter()
        while n < steps and time.perf_counter() - t0 < 5.0:
            ro.step({0: reqs[warm + n]})
            n += 1
        res.update(cpu_requests_per_s=n / (time.perf_counter() - t0), cpu_cores=1, cpu_sample="%d requests" % n)
    return res


def leg_sweep_batched(api, DevicePool, SelectBuffers, stream, with_cpu):
    """Batched sweep: 256 caches of 65,536 blocks in one context, one
    workgroup per cache; one decision (k = 256 per cache) over all of them."""
    import multiprocessing as mp
    import torch
    import synth
    from synth.trace import TRACE_KINDS, TRACE_MU, TRACE_SIGMA
    n_inst, N, k = 256, 65536, 256
    cfg = synth.pool_config("large", n_blocks=N, kinds=TRACE_KINDS, mix=[0.1, 0.4, 0.3, 0.2], mu=TRACE_MU,
                            sigma=TRACE_SIGMA, k=k, max_k=4096, chain_len=128)
    pool = synth.make_pool(cfg, n_blocks=N, seed=1005)
    c = make_cache(api, DevicePool, SelectBuffers, cfg, pool, n_inst=n_inst)
    reps = 20
    with torch.cuda.stream(stream):
        for _ in range(3):
            c["out"].run(c["ctx"], c["now"], k, api.SS_ENGINE_BATCHED, stream=stream)
        with Timer(stream) as t:
            for _ in range(reps):
                c["out"].run(c["ctx"], c["now"], k, api.SS_ENGINE_BATCHED, stream=stream)
    api.sae_destroy(c["ctx"])
    us = t.ms * 1e3 / reps
    alg = BYTES_PER_BLOCK * n_inst * N
    res = dict(workload="256 caches x 65,536 blocks, 4 queues, k=256 per cache, batched engine (one workgroup "
                        "per cache)", gpu_decision_us=us, gpu_blocks_per_s=n_inst * N / (us * 1e-6),
               roofline={"kernel": "k_batched", "bound": "hbm", "achieved": alg / (us * 1e-6) / 1e9,
                         "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": alg / (us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                         "bytes_alg": alg})
    tr = measured_traffic("k_batched_sweep_traffic.json")
    res["roofline"]["traffic"] = tr.get("bytes_per_launch") if tr else None
    if with_cpu:
        n_proc = min(16, cores())
        jobs = [(cfg, 1005, k)] * n_proc
        ctx = mp.get_context("spawn")
        with ctx.Pool(n_proc) as p:
            t0 = time.perf_counter()
            times = p.map(_oracle_select_instance, jobs)
            el = time.perf_counter() - t0
        per = sum(times) / len(times)
        res.update(cpu_cache_select_ms=per * 1e3, cpu_cores=n_proc, cpu_model=cpu_model(),
                   cpu_blocks_per_s=N * n_proc / max(times),
                   cpu_sample="%d caches in %d processes, one per core (%.1f s wall with start-up)" % (
                       n_proc, n_proc, el))
    return res


def sweep_child(name):
    """Child process: one full-length batched-sweep replay (10,000 requests on
    each of 256 caches) with fixed (learn 0) or learned (Algorithms 2 and 3)
    weights; prints the totals per half."""
    import torch
    from paper_2605_18825_amd.engine import DeviceBackend
    from synth.replay import Replay
    from synth.trace import TRACE_CONFIGS, TRACE_KINDS, TRACE_MU, TRACE_ROLES, TRACE_SIGMA, trace_gens
    learn = {"fixed": 0, "learned": 3}[name]
    cfg = TRACE_CONFIGS["batched_sweep"]
    n = cfg["n_inst"]
    gens = trace_gens("batched_sweep", n)
    dev = DeviceBackend(n, cfg["capacity"], TRACE_KINDS, TRACE_ROLES, cfg["max_k"], TRACE_MU, TRACE_SIGMA, cfg["K"],
                        learn)
    rep = Replay(dev, n, cfg["capacity"], cfg["k_min"], cfg["max_k"], cfg["concurrency"])
    t0 = time.perf_counter()
    with torch.cuda.stream(dev.stream):
        for s in range(cfg["n_requests"]):
            rep.step({i: g.next() for i, g in enumerate(gens)})
            if (s + 1) % 1000 == 0:
                print("sweep %s: %d steps (%.0f s)" % (name, s + 1, time.perf_counter() - t0), file=sys.stderr,
                      flush=True)
    dev.close()
    half = n // 2
    out = {cfg["mixes"][0]: rep.summary(list(range(half))), cfg["mixes"][1]: rep.summary(list(range(half, n))),
           "seconds": time.perf_counter() - t0}
    print(json.dumps(out), flush=True)


def leg_sweep_comparison():
    procs = {n: subprocess.Popen([sys.executable, "-u", os.path.abspath(__file__), "--sweep-run", n],
                                 stdout=subprocess.PIPE, text=True) for n in ("fixed", "learned")}
    out = {}
    for n, p in procs.items():
        so, _ = p.communicate(timeout=900)
        if p.returncode != 0:
            raise RuntimeError("sweep child %s failed (%d)" % (n, p.returncode))
        out[n] = json.loads(so.strip().splitlines()[-1])
    res = {"requests_per_cache": 10000, "caches": 256, "seconds": max(out[n]["seconds"] for n in out)}
    for h in ("single_turn_dominant", "multi_turn_dominant"):
        f, l = out["fixed"][h], out["learned"][h]
        res[h] = dict(block_hit_ratio_fixed=f["block_hit_ratio"], block_hit_ratio_learned=l["block_hit_ratio"],
                      prefill_tokens_fixed=f["prefill_tokens"], prefill_tokens_learned=l["prefill_tokens"],
                      prefill_tokens_saved=f["prefill_tokens"] - l["prefill_tokens"])
    return res


# ---------------------------------------------------------------------------- main
def predictor_leg(api, args, R, stream):
    """Session predictor (Sec. 3.3) on 4,096 last-token hidden states of
    d = 4,096, rotating over R batches (256 MB, beyond the last-level cache)."""
    import numpy as np
    import torch
    from synth import predictor as SP
    PN, PD = 4096, 4096
    h0 = SP.hidden_states(PN, PD, 5).view(np.int16)
    hbat = [torch.as_tensor(h0).cuda() for _ in range(R)]
    wnp = SP.weights(PD, 6)
    wp = {kk: torch.as_tensor(v.view(np.int16) if kk == "w1" else v).cuda() for kk, v in wnp.items()}
    pwork = torch.empty((4, PN, 256), dtype=torch.float32, device="cuda")
    plogit = torch.empty(PN, dtype=torch.float32, device="cuda")
    ppred = torch.empty(PN, dtype=torch.uint8, device="cuda")
    with torch.cuda.stream(stream):
        for i in range(args.warmup):
            api.sae_predict_sessions(hbat[i % R], wp, pwork, plogit, ppred, stream=stream)
        with Timer(stream) as tp:
            for i in range(args.steps):
                api.sae_predict_sessions(hbat[i % R], wp, pwork, plogit, ppred, stream=stream)
    ms_pred = tp.ms / args.steps
    pred_bytes = PN * PD * 2 + 256 * PD * 2 + PN * 5  # hidden states, W1, logits and predictions
    pred_flops = 2.0 * PN * PD * 256 + 2.0 * PN * 256 * 64 + 2.0 * PN * 64
    del hbat
    return ms_pred, pred_bytes, pred_flops, PN, PD


def calib_copy(mib):
    """A plain device-to-device copy of `mib` MiB, 4 times: the known-size
    kernel that HBM byte counters are scaled by."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(4):
        dst.copy_(src)
    torch.cuda.synchronize()
    return n * 4


def extra_legs(v):
    """JSON entries of the legs beside the headline, from main()'s measurements `v`."""
    N, HBM_PEAK = v["N"], HBM_PEAK_GBS
    ms_casc, ms_all, ms_ss, ss_steps, ss_per, dc_min = (v[x] for x in ("ms_casc", "ms_all", "ms_ss", "ss_steps",
                                                                         "ss_per", "dc_min"))
    ms_two = v["ms_two"]
    ms_pred, pred_bytes, pred_flops, PN, PD = (v[x] for x in ("ms_pred", "pred_bytes", "pred_flops", "PN", "PD"))
    return {
        "step_two_calls": {
            "value": N / (ms_two * 1e-3) / 1e9, "unit": "G blk/s", "ms_per_step": ms_two,
            "step": "the headline step with sae_prefix_match and sae_score_select as two calls (the selection's "
                    "sampling and bounds after the prefix match instead of in its launch)",
        },
        "score_select_cascade": {
            "value": N / (ms_casc * 1e-3) / 1e9, "unit": "G blk/s", "ms_per_call": ms_casc,
            "decision": "Algorithm 1 one victim at a time (SAE_SS_CASCADE)",
        },
        "all_learners": {
            "value": N / (ms_all * 1e-3) / 1e9, "unit": "G blk/s", "ms_per_step": ms_all,
            "step": "the same step with Algorithms 2, 3, 4 and the decay-power learner on "
                    "(prefix match records reuse intervals)",
        },
        "steady_state": {
            "value": N / (ms_ss * 1e-3) / 1e9, "unit": "G blk/s", "ms_per_step": ms_ss, "steps": ss_steps,
            "last_decision_size": dc_min,
            "note": "the step plus Add() of k fresh blocks into the freed slots (the pool stays full); %d steps "
                    "per cache, so each cache's index is rebuilt from its deleted slots %d times and its "
                    "recently-evicted table as often as its size calls for" % (ss_per, ss_per // 256),
        },
        "step_steady_pools": {
            "value": N / (v["ms_st2"] * 1e-3) / 1e9, "unit": "G blk/s", "ms_per_step": v["ms_st2"],
            "evict_first_share_of_decision": v["ef_share"],
            "step": "the headline step on the pools the steady-state leg left (clusters of equal keys); the "
                    "evict-first queue then supplies only this share of each decision, the rest is Algorithm "
                    "1's second stage",
        },
        "predictor": {
            "value": PN / (ms_pred * 1e-3), "unit": "predictions/s", "ms_per_call": ms_pred,
            "batch": PN, "d": PD,
            "roofline": {"bound": "hbm", "achieved": pred_bytes / (ms_pred * 1e-3) / 1e9, "peak": HBM_PEAK,
                         "unit": "GB/s", "frac": pred_bytes / (ms_pred * 1e-3) / 1e9 / HBM_PEAK,
                         "mfma_tflops_bf16": pred_flops / (ms_pred * 1e-3) / 1e12, "mfma_peak_bf16": 2500.0},
        },
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--replicas", type=int, default=8)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-configs", action="store_true", help="skip the other configurations' legs")
    ap.add_argument("--no-sweep", action="store_true", help="skip the full-length fixed/learned sweep comparison")
    ap.add_argument("--main-only", action="store_true",
                    help="time only the full steps and the score+select pass (for profiler runs)")
    ap.add_argument("--batched-only", action="store_true",
                    help="time only the batched-sweep decision (for profiler runs)")
    ap.add_argument("--predictor-only", action="store_true",
                    help="time only the session predictor (for profiler runs)")
    ap.add_argument("--sweep-run", default=None, help=argparse.SUPPRESS)
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after the timed region, copy this many MiB device-to-device 4 times "
                         "(a plain copy of known size for calibrating HBM byte counters)")
    args = ap.parse_args()
    if args.sweep_run:
        sweep_child(args.sweep_run)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path, so --gpus must be 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    from paper_2605_18825_amd import api
    from paper_2605_18825_amd.pool import DevicePool, SelectBuffers

    torch.cuda.set_device(0)
    if args.predictor_only:
        stream = torch.cuda.Stream()  # default priority
        ms_pred, pred_bytes, pred_flops, PN, PD = predictor_leg(api, args, max(1, args.replicas), stream)
        out = {"predictor": {"ms_per_call": ms_pred, "batch": PN, "d": PD, "bytes_alg": pred_bytes}}
        if args.calib_copy_mib > 0:
            out["calib_copy_bytes"] = calib_copy(args.calib_copy_mib)
        print(json.dumps(out), flush=True)
        return
    if args.batched_only:
        stream = torch.cuda.Stream()  # default priority
        out = {"batched_sweep": leg_sweep_batched(api, DevicePool, SelectBuffers, stream, False)}
        if args.calib_copy_mib > 0:
            out["calib_copy_bytes"] = calib_copy(args.calib_copy_mib)
        print(json.dumps(out), flush=True)
        return
    extra = not args.main_only
    cfg = synth.pool_config("large")
    pool = synth.make_pool(cfg)
    N, Q, k = pool["n_blocks"], len(cfg["kinds"]), cfg["k"]
    reqs, lens = synth.make_requests(pool["chains"], cfg["n_req"], cfg["req_len"], cfg["hit_frac"], cfg["seed"] + 1)
    R = max(1, args.replicas)
    caches = [make_cache(api, DevicePool, SelectBuffers, cfg, pool, max_requests=int(len(lens))) for _ in range(R)]
    d_reqs = torch.as_tensor(np.asarray(reqs, np.uint64).view(np.int64)).cuda()
    d_lens = torch.as_tensor(lens).cuda()
    d_ml = torch.zeros(len(lens), dtype=torch.int32, device="cuda")
    d_ml2 = torch.zeros(len(lens), dtype=torch.int32, device="cuda")
    d_mid = torch.empty((len(lens), reqs.shape[1]), dtype=torch.int32, device="cuda")
    stream = torch.cuda.Stream()  # default priority
    stream_b = torch.cuda.Stream()  # default priority
    torch.cuda.synchronize()

    def step(i):
        c = caches[i % R]
        c["out"].run_after_match(c["ctx"], d_reqs, d_lens, c["now"], api.PM_TOUCH | api.PM_STATS, d_ml, c["now"], k,
                                 api.SS_COMMIT, stream=stream)
        api.sae_feedback_update(c["ctx"], 0, stream=stream)
        c["now"] += 1000

    def step_two_calls(i):
        c = caches[i % R]
        api.sae_prefix_match(c["ctx"], d_reqs, d_lens, c["now"], api.PM_TOUCH | api.PM_STATS, d_ml, stream=stream)
        c["out"].run(c["ctx"], c["now"], k, api.SS_COMMIT, stream=stream)
        api.sae_feedback_update(c["ctx"], 0, stream=stream)
        c["now"] += 1000

    def step_all_learners(i):
        c = caches[i % R]
        c["out"].run_after_match(c["ctx"], d_reqs, d_lens, c["now"], api.PM_TOUCH | api.PM_STATS | api.PM_INTERVALS,
                                 d_ml, c["now"], k, api.SS_COMMIT, matched_ids=d_mid, stream=stream)
        api.sae_feedback_update(c["ctx"], 0, stream=stream)
        c["now"] += 1000

    def timed_loop(fn, n, w):
        for i in range(w):
            fn(i)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(n):
            fn(w + i)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3 / n

    with torch.cuda.stream(stream):
        # --- full steps (the headline)
        for i in range(args.warmup):
            step(i)
        torch.cuda.synchronize()
        for c in caches:
            api.sae_profile_enable(c["ctx"], True)
            api.sae_profile_read(c["ctx"])
        t0 = time.perf_counter()
        for i in range(args.steps):
            step(args.warmup + i)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        scan_ms, scan_n = 0.0, 0
        for c in caches:
            ms, n = api.sae_profile_read(c["ctx"])
            api.sae_profile_enable(c["ctx"], False)
            scan_ms += ms
            scan_n += n
        note("full steps: %.3f ms/step" % ((t1 - t0) * 1e3 / args.steps))
        # --- score+select alone (no commit), each pass bracketed by HIP events on its stream
        for i in range(args.warmup):
            caches[i % R]["out"].run(caches[i % R]["ctx"], caches[i % R]["now"], k, 0, stream=stream)
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        s0 = time.perf_counter()
        for i in range(args.steps):
            c = caches[i % R]
            evs[i][0].record(stream)
            c["out"].run(c["ctx"], c["now"], k, 0, stream=stream)
            evs[i][1].record(stream)
        torch.cuda.synchronize()
        s1 = time.perf_counter()
        pass_ms = sum(a.elapsed_time(b) for a, b in evs) / args.steps
        if extra:
            # --- the same pass with a read-only prefix match on a second stream
            def pair(i, sel=True, pm=True):
                c = caches[i % R]
                if sel:
                    c["out"].run(c["ctx"], c["now"], k, 0, stream=stream)
                if pm:
                    api.sae_prefix_match(c["ctx"], d_reqs, d_lens, c["now"], 0, d_ml2, stream=stream_b)
            note("score+select alone: %.3f ms/pass" % pass_ms)
            ms_pm_alone = timed_loop(lambda i: pair(i, sel=False), args.steps, args.warmup)
            ms_pair = timed_loop(pair, args.steps, args.warmup)
            # --- the headline step issued as two calls
            ms_two = timed_loop(step_two_calls, args.steps, args.warmup)
            # --- cascading decision (Algorithm 1 one victim at a time)
            ms_casc = timed_loop(lambda i: caches[i % R]["out"].run(caches[i % R]["ctx"], caches[i % R]["now"], k,
                                                                    api.SS_CASCADE, stream=stream), args.steps, args.warmup)
            # --- every learner on: Algorithms 2, 3, 4 and the decay power, the prefix match recording reuse intervals
            for c in caches:
                api.sae_set_params(c["ctx"], -1, api.make_params(Q, mu=cfg["mu"], sigma=cfg["sigma"], K=k, learn=15),
                                   stream=stream)
            ms_all = timed_loop(step_all_learners, args.steps, args.warmup)
            for c in caches:
                api.sae_set_params(c["ctx"], -1, api.make_params(Q, mu=cfg["mu"], sigma=cfg["sigma"], K=k), stream=stream)
            note("pair, cascade, all learners done")
            # --- steady state: each step also inserts k fresh blocks into the slots its decision freed
            # (Add(), so the pool stays full), over enough steps per cache that the index (rebuilt
            # every 256 commits of k) and recently-evicted tables are rebuilt as in a long run
            ss_per = 1040
            ss_steps = R * ss_per
            now0 = max(c["now"] for c in caches)
            for c in caches:
                c["now"] = now0
            gen = torch.Generator(device="cuda")
            gen.manual_seed(7)
            ins_hash = torch.randint(1, 1 << 62, (ss_per, k), dtype=torch.int64, device="cuda", generator=gen)
            ins_la = (now0 + 1000 * torch.arange(ss_per, dtype=torch.int32, device="cuda"))[:, None].expand(
                ss_per, k).contiguous()
            ins_meta = caches[0]["dp"].meta[:k].clone()  # queue, type and num_tokens of k pool blocks
            ins_off = caches[0]["dp"].off[:k].clone()
            ins_parent = torch.full((k,), -1, dtype=torch.int32, device="cuda")
            torch.cuda.synchronize()

            def step_insert(i):
                c = caches[i % R]
                n = i // R
                step(i)
                api.sae_insert_blocks(c["ctx"], c["out"].decision[0, :k], ins_hash[n], ins_parent, ins_la[n], ins_meta,
                                      ins_off, stream=stream)
                if (i + 1) % 2000 == 0:
                    note("steady state: %d of %d steps issued" % (i + 1, ss_steps))

            ms_ss = timed_loop(step_insert, ss_steps, 0)
            dc_min = min(int(c["out"].decision_count[0]) for c in caches)
            # --- the headline step on the steady-state pools (no Add()): most of each decision now comes
            # from Algorithm 1's second stage, and the pools hold clusters of equal keys
            ms_st2 = timed_loop(step, args.steps, args.warmup)
            ef_share = sum(int(c["out"].count[0, 0]) for c in caches) / float(k * len(caches))
    if extra:
        note("steady state: %.3f ms/step over %d steps" % (ms_ss, ss_steps))
        ms_pred, pred_bytes, pred_flops, PN, PD = predictor_leg(api, args, R, stream)
    else:
        note("score+select alone: %.3f ms/pass" % pass_ms)
    st = 0
    for c in caches:
        st |= api.sae_poll_status(c["ctx"])
    bad = [s for s in api.status_names(st) if s not in ("SELECT_FALLBACK",)]
    if bad:
        print("device status: %s" % bad, file=sys.stderr)

    ms_step = (t1 - t0) * 1e3 / args.steps
    ms_sel = (s1 - s0) * 1e3 / args.steps
    scan_avg_ms = scan_ms / max(scan_n, 1)
    alg_bytes = BYTES_PER_BLOCK * N
    achieved = alg_bytes / (pass_ms * 1e-3) / 1e9
    traffic = measured_traffic()
    line = {
        "metric": METRIC,
        "value": N / (ms_step * 1e-3) / 1e9,
        "unit": "G blk/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "one 4,194,304-block cache, 5 queues, k=4096; step = prefix match of 4096x128 hashes "
                        "+ score/select/commit (one sae_match_select call) + feedback",
            "blocks": N, "queues": Q, "k": k, "requests": int(len(lens)), "hashes_per_request": int(reqs.shape[1]),
            "replicas": R,
        },
        "roofline": {
            "kernel": "score+select pass (k_sample, k_split, k_scan, k_final)", "bound": "hbm",
            "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic.get("pass_bytes_per_call") if traffic else None, "avg_pass_ms": pass_ms,
            "bytes_per_pass_alg": alg_bytes,
            "scan_kernel": {
                "kernel": "k_scan", "achieved": alg_bytes / (scan_avg_ms * 1e-3) / 1e9,
                "frac": alg_bytes / (scan_avg_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, "avg_launch_ms": scan_avg_ms,
                "launches": scan_n, "traffic": traffic.get("scan_bytes_per_launch") if traffic else None,
            },
        },
        "score_select": {
            "value": N / (ms_sel * 1e-3) / 1e9, "unit": "G blk/s", "ms_per_call": ms_sel, "ms_per_pass_events": pass_ms,
            "hbm_frac_at_10B_per_block": alg_bytes / (pass_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
        },
        "device_status": api.status_names(st),
    }
    if extra:
        line["score_select"]["with_concurrent_prefix_match"] = {
            "ms_pair": ms_pair, "ms_prefix_match_alone": ms_pm_alone, "ms_score_select_alone": ms_sel,
            "requests": int(len(lens)), "hashes_per_request": int(reqs.shape[1]),
            "note": "read-only prefix match on a second stream of the same context",
        }
        line.update(extra_legs(locals()))
    for c in caches:
        api.sae_destroy(c["ctx"])
    del caches
    torch.cuda.synchronize()
    if args.calib_copy_mib > 0:
        line["calib_copy_bytes"] = calib_copy(args.calib_copy_mib)
    if not args.no_configs and extra:
        line["configs"] = {}
        for name, fn in (("tiny", lambda: leg_tiny(api, DevicePool, SelectBuffers, stream, not args.no_cpu)),
                         ("mid", lambda: leg_mid(api, DevicePool, SelectBuffers, stream, not args.no_cpu)),
                         ("trace_balanced", lambda: leg_trace(stream, not args.no_cpu)),
                         ("batched_sweep",
                          lambda: leg_sweep_batched(api, DevicePool, SelectBuffers, stream, not args.no_cpu))):
            line["configs"][name] = fn()
            note("config %s done" % name)
        if not args.no_sweep:
            line["configs"]["batched_sweep"]["fixed_vs_learned"] = leg_sweep_comparison()
            note("sweep comparison done")
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(cfg, pool, reqs, lens, args.cpu_seconds)
        note("cpu baseline done")
        line["cpu_baseline"]["recency_lists"] = cpu_recency_lists(cfg, pool)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
