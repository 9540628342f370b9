"""Benchmark of the eviction hot path on one MI355X.

Workload: one cache of 4,194,304 blocks (64M tokens), 5 queues (evict-first,
structural, chat log-normal, agent log-normal, recency), k = 4,096 victims per
queue, and a batch of 4,096 prefix-match requests of 128 block hashes.

A step is one full pass of the hot path on one cache:
  sae_prefix_match (touch + stats) -> sae_score_select (every block scored,
  per-queue k smallest, Algorithm 1 decision, commit) -> sae_feedback_update.
Steps rotate over R independent caches (own pool, index and recently-evicted
table) so that the working set exceeds the 256 MB last-level cache and the
pool is read from HBM.

value = blocks scored+selected per second over the timed steps (G blk/s).
The JSON line also carries the score+select call alone, the roofline of the
scoring kernel (bytes per block x blocks / its HIP-event-timed duration) and
the CPU oracle timed on a bounded sample on the host.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "cached blocks scored+selected per sec (G blk/s) at 4M blocks; % HBM peak"
HBM_PEAK_GBS = 8000.0
BYTES_PER_BLOCK = 10  # last_access 4 + meta 2 + off 4: what the scoring pass must read
SCAN_KERNEL_SOURCES = ["paper_2605_18825_amd/csrc/k_select.hip", "paper_2605_18825_amd/csrc/sae_internal.h"]


def kernel_source_hash():
    h = hashlib.sha256()
    for f in SCAN_KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic():
    """HBM bytes per launch of the scoring kernel from rocprofv3 counters, if the
    committed measurement was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", "k_scan_large_pool_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    return t.get("bytes_per_launch")


def cpu_baseline(cfg, pool, reqs, lens, budget_s):
    """The oracle as it stands, single-threaded on the host, on a bounded number
    of full steps of the same workload."""
    import numpy as np
    import oracle
    prm = oracle.Params(len(cfg["kinds"]), mu=cfg["mu"], sigma=cfg["sigma"], K=cfg["k"])
    oc = oracle.OracleCache(pool["n_blocks"], cfg["kinds"], prm)
    oc.bind(pool["last_access"], pool["queue"], oracle.block_type(pool["counts"]), pool["ntok"], pool["ob"],
            pool["omax"], pool["valid"], pool["ref_count"], pool["parent"], pool["hash"], pool["access_count"])
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
    """Part of the CPU baseline leg: a faster exact CPU selection (per-(queue, type) recency lists, the
    per-queue heap idea) on the same pool: score+select without commit, timed
    apart from building the lists (which a live cache keeps up incrementally);
    the oracle's full-sort selection of the same call is timed beside it and
    the two decisions are compared."""
    import numpy as np
    import oracle
    from oracle.recency import RecencyLists
    prm = oracle.Params(len(cfg["kinds"]), mu=cfg["mu"], sigma=cfg["sigma"], K=cfg["k"])
    oc = oracle.OracleCache(pool["n_blocks"], cfg["kinds"], prm)
    oc.bind(pool["last_access"], pool["queue"], oracle.block_type(pool["counts"]), pool["ntok"], pool["ob"],
            pool["omax"], pool["valid"], pool["ref_count"], pool["parent"], pool["hash"], pool["access_count"])
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--replicas", type=int, default=8)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after the timed region, copy this many MiB device-to-device 4 times "
                         "(a plain copy of known size for calibrating HBM byte counters)")
    args = ap.parse_args()
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
    cfg = synth.pool_config("large")
    pool = synth.make_pool(cfg)
    N, Q, k = pool["n_blocks"], len(cfg["kinds"]), cfg["k"]
    reqs, lens = synth.make_requests(pool["chains"], cfg["n_req"], cfg["req_len"], cfg["hit_frac"], cfg["seed"] + 1)
    R = max(1, args.replicas)
    caches = []
    for r in range(R):
        ctx = api.sae_create(1, N, cfg["kinds"], max_k=k, max_requests=int(len(lens)))
        dp = DevicePool(1, N)
        dp.fill_instance(0, pool)
        dp.bind(ctx)
        api.sae_index_build(ctx)
        api.sae_set_params(ctx, -1, api.make_params(Q, mu=cfg["mu"], sigma=cfg["sigma"], K=k))
        caches.append(dict(ctx=ctx, dp=dp, out=SelectBuffers(1, Q, k), now=pool["now"]))
    d_reqs = torch.as_tensor(np.asarray(reqs, np.uint64).view(np.int64)).cuda()
    d_lens = torch.as_tensor(lens).cuda()
    d_ml = torch.zeros(len(lens), dtype=torch.int32, device="cuda")
    d_mid = torch.empty((len(lens), reqs.shape[1]), dtype=torch.int32, device="cuda")
    stream = torch.cuda.Stream()  # default priority
    torch.cuda.synchronize()

    def step(i):
        c = caches[i % R]
        api.sae_prefix_match(c["ctx"], d_reqs, d_lens, c["now"], api.PM_TOUCH | api.PM_STATS, d_ml, stream=stream)
        c["out"].run(c["ctx"], c["now"], k, api.SS_COMMIT, stream=stream)
        api.sae_feedback_update(c["ctx"], 0, stream=stream)
        c["now"] += 1000

    def select_only(i):
        c = caches[i % R]
        c["out"].run(c["ctx"], c["now"], k, 0, stream=stream)

    def select_cascade(i):
        c = caches[i % R]
        c["out"].run(c["ctx"], c["now"], k, api.SS_CASCADE, stream=stream)

    def step_all_learners(i):
        c = caches[i % R]
        api.sae_prefix_match(c["ctx"], d_reqs, d_lens, c["now"], api.PM_TOUCH | api.PM_STATS | api.PM_INTERVALS,
                             d_ml, matched_ids=d_mid, stream=stream)
        c["out"].run(c["ctx"], c["now"], k, api.SS_COMMIT, stream=stream)
        api.sae_feedback_update(c["ctx"], 0, stream=stream)
        c["now"] += 1000

    with torch.cuda.stream(stream):
        # --- full steps
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
        # --- score+select alone (no commit), same rotation
        for i in range(args.warmup):
            select_only(i)
        torch.cuda.synchronize()
        s0 = time.perf_counter()
        for i in range(args.steps):
            select_only(i)
        torch.cuda.synchronize()
        s1 = time.perf_counter()
        # --- score+select with a cascading decision (Algorithm 1 one victim at a time)
        for i in range(args.warmup):
            select_cascade(i)
        torch.cuda.synchronize()
        c0 = time.perf_counter()
        for i in range(args.steps):
            select_cascade(i)
        torch.cuda.synchronize()
        c1 = time.perf_counter()
        # --- the same step with every learner on: Algorithms 2, 3, 4 and the
        # decay power, the prefix match recording reuse intervals
        for c in caches:
            api.sae_set_params(c["ctx"], -1, api.make_params(Q, mu=cfg["mu"], sigma=cfg["sigma"], K=k, learn=15),
                               stream=stream)
        for i in range(args.warmup):
            step_all_learners(i)
        torch.cuda.synchronize()
        a0 = time.perf_counter()
        for i in range(args.steps):
            step_all_learners(i)
        torch.cuda.synchronize()
        a1 = time.perf_counter()
    # --- session predictor (Sec. 3.3) on 4,096 last-token hidden states of
    # d = 4,096, rotating over 8 batches (256 MB, beyond the last-level cache)
    from synth import predictor as SP
    PN, PD = 4096, 4096
    h0 = SP.hidden_states(PN, PD, 5).view(np.int16)
    hbat = [torch.as_tensor(h0).cuda() for _ in range(R)]
    wnp = SP.weights(PD, 6)
    wp = {k: torch.as_tensor(v.view(np.int16) if k == "w1" else v).cuda() for k, v in wnp.items()}
    pwork = torch.empty((4, PN, 256), dtype=torch.float32, device="cuda")
    plogit = torch.empty(PN, dtype=torch.float32, device="cuda")
    ppred = torch.empty(PN, dtype=torch.uint8, device="cuda")
    with torch.cuda.stream(stream):
        for i in range(args.warmup):
            api.sae_predict_sessions(hbat[i % R], wp, pwork, plogit, ppred, stream=stream)
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        ev0.record(stream)
        for i in range(args.steps):
            api.sae_predict_sessions(hbat[i % R], wp, pwork, plogit, ppred, stream=stream)
        ev1.record(stream)
        torch.cuda.synchronize()
    ms_pred = ev0.elapsed_time(ev1) / args.steps
    pred_bytes = PN * PD * 2 + 256 * PD * 2 + PN * 5  # hidden states, W1, logits and predictions
    pred_flops = 2.0 * PN * PD * 256 + 2.0 * PN * 256 * 64 + 2.0 * PN * 64
    del hbat
    st = 0
    for c in caches:
        st |= api.sae_poll_status(c["ctx"])
    bad = [s for s in api.status_names(st) if s not in ("SELECT_FALLBACK",)]
    if bad:
        print("device status: %s" % bad, file=sys.stderr)

    ms_step = (t1 - t0) * 1e3 / args.steps
    ms_sel = (s1 - s0) * 1e3 / args.steps
    ms_all = (a1 - a0) * 1e3 / args.steps
    ms_casc = (c1 - c0) * 1e3 / args.steps
    scan_avg_ms = scan_ms / max(scan_n, 1)
    alg_bytes = BYTES_PER_BLOCK * N
    achieved = alg_bytes / (scan_avg_ms * 1e-3) / 1e9
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
                        "+ score/select/commit + feedback",
            "blocks": N, "queues": Q, "k": k, "requests": int(len(lens)), "hashes_per_request": int(reqs.shape[1]),
            "replicas": R,
        },
        "score_select": {
            "value": N / (ms_sel * 1e-3) / 1e9, "unit": "G blk/s", "ms_per_call": ms_sel,
            "hbm_frac_at_10B_per_block": BYTES_PER_BLOCK * N / (ms_sel * 1e-3) / 1e9 / HBM_PEAK_GBS,
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
        "predictor": {
            "value": PN / (ms_pred * 1e-3), "unit": "predictions/s", "ms_per_call": ms_pred,
            "batch": PN, "d": PD,
            "roofline": {"bound": "hbm", "achieved": pred_bytes / (ms_pred * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": pred_bytes / (ms_pred * 1e-3) / 1e9 / HBM_PEAK_GBS,
                         "mfma_tflops_bf16": pred_flops / (ms_pred * 1e-3) / 1e12, "mfma_peak_bf16": 2500.0},
        },
        "roofline": {
            "kernel": "k_scan", "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS, "traffic": traffic, "avg_launch_ms": scan_avg_ms,
            "launches": scan_n, "bytes_per_launch_alg": alg_bytes,
        },
        "device_status": api.status_names(st),
    }
    for c in caches:
        api.sae_destroy(c["ctx"])
    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(4):
            dst.copy_(src)
        torch.cuda.synchronize()
        line["calib_copy_bytes"] = n * 4
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(cfg, pool, reqs, lens, args.cpu_seconds)
        line["cpu_baseline"]["recency_lists"] = cpu_recency_lists(cfg, pool)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
