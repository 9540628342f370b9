"""GPU bit-identity of the fp32 scoring recipe on dense grids, through the C
ABI: pools whose blocks carry chosen (dt, o_b, o_max, type) values are scored
with k = all, and every P returned must equal the oracle's bits."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

import torch  # noqa: E402

from harness import Pair, say  # noqa: E402
from paper_2605_18825_amd import api  # noqa: E402

NB = 8192


def grid_pool(n, queue, la, ob, omax, counts=None):
    p = dict(n_blocks=n, now=0, counts=counts if counts is not None else np.tile([[16, 0, 0, 0, 0]], (n, 1)).astype(np.uint8),
             last_access=la.astype(np.int32), access_count=np.zeros(n, np.int32), queue=queue.astype(np.int32),
             ntok=np.full(n, 16, np.int32), ob=ob.astype(np.int32), omax=omax.astype(np.int32),
             valid=np.ones(n, bool), ref_count=np.zeros(n, np.int32), parent=np.full(n, -1, np.int32),
             hash=np.arange(1, n + 1, dtype=np.uint64), chains=None)
    return p


def refill(pair, la, ob=None, omax=None):
    pair.oc.la[:] = la
    pair.dp.last_access.copy_(torch.as_tensor(la.astype(np.int32)))
    if ob is not None:
        pair.oc.ob[:] = ob
        pair.oc.omax[:] = omax
        off = api.off_to_u32(api.pack_off(torch.as_tensor(ob.astype(np.int64)), torch.as_tensor(omax.astype(np.int64))))
        pair.dp.off.copy_(off)


@pytest.mark.parametrize("mu,sigma", [(11.727755, 1.25), (9.187755, 1.34), (8.0, 0.3), (2.0, 4.0)])
def test_lognormal_grid(mu, sigma):
    now = 1 << 30
    z = np.zeros(NB, np.int64)
    pair = Pair([2], grid_pool(NB, z, z, z, z), NB, mu=[mu], sigma=[sigma])
    try:
        dts = np.concatenate([np.arange(0, 1 << 17), np.unique(np.geomspace(1 << 17, 1 << 30, 60000).astype(np.int64))])
        for i in range(0, len(dts), NB):
            dt = dts[i:i + NB]
            if len(dt) < NB:
                dt = np.concatenate([dt, np.full(NB - len(dt), dt[-1])])
            refill(pair, now - dt)
            pair.select(now, NB)
        say("lognormal grid mu=%g sigma=%g: %d dt values bit-identical" % (mu, sigma, len(dts)))
    finally:
        pair.close()


@pytest.mark.parametrize("gamma", [1.0, 0.3, 0.94, 2.5])
def test_structural_grid(gamma):
    now = 1 << 20
    omax = np.repeat(np.arange(0, 300), 301)[:NB * 11]
    ob = np.tile(np.arange(0, 301), 300)[:NB * 11]
    keep = ob <= omax
    ob, omax = ob[keep], omax[keep]
    z = np.zeros(NB, np.int64)
    pair = Pair([1], grid_pool(NB, z, z, z, z), NB, gamma=gamma)
    rng = np.random.default_rng(0)
    try:
        for i in range(0, len(ob), NB):
            o1, o2 = ob[i:i + NB], omax[i:i + NB]
            if len(o1) < NB:
                o1 = np.concatenate([o1, np.zeros(NB - len(o1), np.int64)])
                o2 = np.concatenate([o2, np.zeros(NB - len(o2), np.int64)])
            refill(pair, now - rng.integers(1, 1 << 20, NB), o1, o2)
            pair.select(now, NB)
    finally:
        pair.close()


def test_division_and_subnormal_scores():
    """Recency queue: P = fl(fl(alpha w) / dt); weights down to 1e-38 make P
    subnormal, which must round identically."""
    z = np.zeros(NB, np.int64)
    counts = np.zeros((NB, 5), np.uint8)
    counts[np.arange(NB), np.arange(NB) % 5] = 16
    w = [1e-38, 3.3e-30, 0.1, 1.0, 4.99]
    pair = Pair([3], grid_pool(NB, z, z, z, z, counts=counts), NB, w=w, alpha=[0.7])
    rng = np.random.default_rng(2)
    try:
        now = 1 << 30
        for it in range(40):
            dt = rng.integers(1, 1 << 30, NB) if it % 2 else rng.integers(1, 1 << 12, NB)
            refill(pair, now - dt)
            pair.select(now, NB)
    finally:
        pair.close()


def _dev_eval(fn, x):
    xd = torch.as_tensor(x).cuda()
    yd = torch.empty_like(xd)
    api.sae_recipe_eval(fn, xd, yd)
    torch.cuda.synchronize()
    return yd.cpu().numpy()


def test_elementary_functions_bit_identical():
    """Device ln / exp / erfc against the oracle's transcription of the same
    recipe, on dense grids of float bit patterns."""
    from oracle import _native as dsr
    rng = np.random.default_rng(11)
    lo, hi = np.float32(1.0).view(np.uint32), np.float32(2.0 ** 31).view(np.uint32)
    xs_ln = np.concatenate([np.arange(lo, lo + (1 << 20), dtype=np.uint32),
                            rng.integers(np.float32(1e-30).view(np.uint32), hi, 1 << 21, dtype=np.uint32)]).view(np.float32)
    xs_exp = np.concatenate([np.linspace(-90, 90, 1 << 20, dtype=np.float32),
                             rng.uniform(-87, 88, 1 << 20).astype(np.float32)])
    xs_erfc = np.concatenate([np.arange(0, 1 << 20, dtype=np.uint32).view(np.float32),
                              rng.integers(0, np.float32(9.5).view(np.uint32), 1 << 21, dtype=np.uint32).view(np.float32)])
    for fn, xs, ref in ((api.FN_LN, xs_ln, dsr.ln), (api.FN_EXP, xs_exp, dsr.exp), (api.FN_ERFC, xs_erfc, dsr.erfc)):
        d = _dev_eval(fn, xs)
        o = ref(xs)
        bad = np.flatnonzero(d.view(np.uint32) != o.view(np.uint32))
        assert bad.size == 0, (fn, xs[bad[:5]], d[bad[:5]], o[bad[:5]])
    say("elementary functions: %d inputs bit-identical" % (xs_ln.size + xs_exp.size + xs_erfc.size))


def test_monotonicity_exhaustive():
    """What the scan's pruning of log-normal queues relies on, over EVERY float
    input: ln is non-decreasing on [1, 2^31], and erfc never rises above its
    value at a smaller argument by more than a relative 2^-20 on [0, 9]."""
    chunk = 1 << 25
    # ln, ascending
    lo, hi = int(np.float32(1.0).view(np.uint32)), int(np.float32(2.0 ** 31).view(np.uint32))
    prev = None
    y = torch.empty(chunk, dtype=torch.float32, device="cuda")
    for a in range(lo, hi + 1, chunk):
        b = min(a + chunk, hi + 1)
        x = torch.arange(a, b, dtype=torch.int64, device="cuda").to(torch.int32).view(torch.float32)
        yy = y[:b - a]
        api.sae_recipe_eval(api.FN_LN, x, yy)
        assert bool((yy[1:] >= yy[:-1]).all()), "ln decreases inside [%d, %d)" % (a, b)
        if prev is not None:
            assert float(yy[0]) >= prev, "ln decreases at bits %d" % a
        prev = float(yy[-1])
    # erfc, descending, carrying the largest value at larger arguments
    top = int(np.float32(9.0).view(np.uint32))
    run = 0.0
    worst = 1.0
    b = top + 1
    while b > 0:
        a = max(0, b - chunk)
        x = torch.arange(a, b, dtype=torch.int64, device="cuda").to(torch.int32).view(torch.float32)
        yy = y[:b - a]
        api.sae_recipe_eval(api.FN_ERFC, x, yy)
        suf = torch.flip(torch.cummax(torch.flip(yy, [0]), 0).values, [0])
        suf = torch.clamp(suf, min=run)
        pos = yy > 0
        r = float((suf[pos].double() / yy[pos].double()).max()) if bool(pos.any()) else 1.0
        worst = max(worst, r)
        run = max(run, float(yy.max()))
        b = a
    torch.cuda.synchronize()
    say("monotonicity: ln non-decreasing on [1, 2^31]; erfc worst relative rise %.3e" % (worst - 1.0))
    assert worst - 1.0 <= 2.0 ** -20
