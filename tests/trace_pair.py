"""Trace replay on the HIP path and on the oracle side by side (GPU tests).

Both replays get the same requests from synth.trace; each uses only its own
backend's outputs.  After every step the match lengths and the eviction
decisions of the instances the oracle replays are compared element by
element; counters, learned weights and pool state are compared every
`check_every` steps and at the end."""
import numpy as np
import torch

from harness import say
from oracle_backend import OracleBackend
from paper_2605_18825_amd import api
from paper_2605_18825_amd.engine import DeviceBackend
from synth.replay import Replay
from synth.trace import TRACE_CONFIGS
from trace_setup import KINDS, MU, ROLES, SIGMA, trace_gens  # noqa: F401


def check_pool(dev, orc, i):
    torch.cuda.synchronize()
    N = dev.N
    sl = slice(i * N, (i + 1) * N)
    o = orc.c[i]
    m = api.unpack_meta(dev.pool.meta[sl])
    valid = m["valid"].cpu().numpy()
    assert np.array_equal(valid, o.valid), "instance %d: valid bits differ" % i
    v = o.valid
    for name, got, want in (
            ("leaf", m["leaf"].cpu().numpy(), o.child_count == 0),
            ("ref", m["ref"].cpu().numpy(), o.ref_count > 0),
            ("queue", m["queue"].cpu().numpy(), o.queue),
            ("tau", m["tau"].cpu().numpy(), o.tau),
            ("child_count", dev.pool.child_count[sl].cpu().numpy(), o.child_count),
            ("ref_count", dev.pool.ref_count[sl].cpu().numpy(), o.ref_count),
            ("last_access", dev.pool.last_access[sl].cpu().numpy(), o.la),
            ("access_count", dev.pool.access_count[sl].cpu().numpy(), o.access_count),
            ("hash", dev.pool.hash[sl].cpu().numpy().view(np.uint64), o.hash)):
        assert np.array_equal(np.asarray(got)[v], np.asarray(want)[v]), "instance %d: %s differs" % (i, name)


def check_state(dev, orc, i):
    cd, co = dev.counters(i), orc.counters(i)
    for key in ("evicted", "missed", "hits", "evictions", "ev_count", "pending", "n_updates", "bin_hits", "bin_missed",
                "type_hits", "type_added", "resident"):
        assert cd[key] == co[key], "instance %d: %s %s vs oracle %s" % (i, key, cd[key], co[key])
    (wd, ad), (wo, ao) = dev.params(i), orc.params(i)
    assert np.array_equal(wd.view(np.uint32), wo.view(np.uint32)), "instance %d: w %s vs %s" % (i, wd, wo)
    assert np.array_equal(ad.view(np.uint32), ao.view(np.uint32)), "instance %d: alpha %s vs %s" % (i, ad, ao)
    (md, sd, gd), (mo, so, go) = dev.timing_params(i), orc.timing_params(i)
    assert np.array_equal(md.view(np.uint32), mo.view(np.uint32)), "instance %d: mu %s vs %s" % (i, md, mo)
    assert np.array_equal(sd.view(np.uint32), so.view(np.uint32)), "instance %d: sigma %s vs %s" % (i, sd, so)
    assert gd.view(np.uint32) == go.view(np.uint32), "instance %d: gamma %r vs %r" % (i, gd, go)


def run_pair(name, steps, oracle_insts, n_inst=None, capacity=None, learn=3, check_every=100, w=1.0, cascade=False,
             **gen_over):
    cfg = TRACE_CONFIGS[name]
    n_inst = cfg["n_inst"] if n_inst is None else n_inst
    capacity = cfg["capacity"] if capacity is None else capacity
    gens = trace_gens(name, n_inst, **gen_over)
    dev = DeviceBackend(n_inst, capacity, KINDS, ROLES, cfg["max_k"], MU, SIGMA, cfg["K"], learn, w=w, cascade=cascade)
    orc = OracleBackend(oracle_insts, capacity, KINDS, ROLES, MU, SIGMA, cfg["K"], learn, w=w, cascade=cascade)
    rd = Replay(dev, n_inst, capacity, cfg["k_min"], cfg["max_k"], cfg["concurrency"])
    ro = Replay(orc, n_inst, capacity, cfg["k_min"], cfg["max_k"], cfg["concurrency"], insts=oracle_insts)
    try:
        for s in range(steps):
            reqs = {i: g.next() for i, g in enumerate(gens)}
            a = rd.step(reqs)
            b = ro.step({i: reqs[i] for i in oracle_insts})
            for i in oracle_insts:
                (mla, da), (mlb, db) = a[i], b[i]
                assert mla == mlb, "step %d instance %d: match length %d vs oracle %d" % (s, i, mla, mlb)
                assert len(da) == len(db), "step %d instance %d: %d decisions vs oracle %d" % (s, i, len(da), len(db))
                for r, (x, y) in enumerate(zip(da, db)):
                    if not np.array_equal(x, y):
                        raise AssertionError("step %d instance %d decision %d: %d victims vs oracle %d, first "
                                             "difference %s" % (s, i, r, len(x), len(y),
                                                                np.nonzero(x[:min(len(x), len(y))] !=
                                                                           y[:min(len(x), len(y))])[0][:3]))
            if s % check_every == 0 or s == steps - 1:
                say("%s step %d: %s" % (name, s, rd.summary(oracle_insts)))
                for i in oracle_insts:
                    check_state(dev, orc, i)
        for i in oracle_insts:
            check_pool(dev, orc, i)
        st = dev.status()
        assert set(st) <= {"SELECT_FALLBACK"}, st
        return rd, ro, dev
    finally:
        dev.close()
