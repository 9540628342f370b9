"""What the learners converge to on the synthetic mixes (Table 2's single-
turn-dominant and multi-turn-dominant traffic, 36K-token caches, the paper's
initial token weights 2.0 / 1.5 / 1.0 / 1.0 / 0.1), against the orderings the
paper reports in Sec. 5: token weights system > user > tool, response >
chain-of-thought (Algorithm 3), and queue weights that favour the multi-turn
queues under multi-turn-dominant traffic and the structural queue under
single-turn-dominant traffic (both queue rules; the paper's 24:1 and 1:8 come
from its own traces).  One replay of 32 caches: Algorithms 2/3/4 and gamma on
16 of them, the appendix text's token and queue rules on the other 16.
GPU only: parity of every step with the oracle is in test_gpu_trace.py."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

from harness import say  # noqa: E402
from paper_2605_18825_amd import api  # noqa: E402
from paper_2605_18825_amd.engine import DeviceBackend  # noqa: E402
from synth.replay import Replay  # noqa: E402
from synth.trace import TraceGen  # noqa: E402
from trace_pair import KINDS, MU, ROLES, SIGMA  # noqa: E402

SYS, USER, TOOL, RESP, COT = range(5)
STRUCT, CHAT, AGENT = 1, 2, 3
ALGS = api.LEARN_TOKEN_WEIGHTS | api.LEARN_QUEUE_WEIGHTS | api.LEARN_LOGNORMAL | api.LEARN_DECAY_POWER
TEXT = api.LEARN_TOKEN_EMA | api.LEARN_QUEUE_REL | api.LEARN_LOGNORMAL | api.LEARN_DECAY_POWER


def test_learned_orderings_on_the_two_mixes():
    n, steps = 32, 3000
    mixes = (["single_turn_dominant"] * 8 + ["multi_turn_dominant"] * 8) * 2
    gens = [TraceGen(mixes[i], 7000 + i) for i in range(n)]
    w0 = list(api.PAPER_INIT_W)
    dev = DeviceBackend(n, 2250, KINDS, ROLES, 1024, MU, SIGMA, 32, ALGS, w=w0)
    try:
        for i in range(16, 32):
            api.sae_set_params(dev.ctx, i, api.make_params(4, w=w0, mu=MU, sigma=SIGMA, K=32, learn=TEXT))
        rd = Replay(dev, n, 2250, 1, 1024, 4)
        for s in range(steps):
            rd.step({i: g.next() for i, g in enumerate(gens)})
            if s % 1000 == 0:
                say("orderings: step %d" % s)
        W = np.array([dev.params(i)[0] for i in range(n)])
        A = np.array([dev.params(i)[1] for i in range(n)])
        res = {}
        for rules, lo in (("algorithms", 0), ("text", 16)):
            for mix, sl in (("single", slice(lo, lo + 8)), ("multi", slice(lo + 8, lo + 16))):
                res[rules, mix] = (W[sl].mean(0), A[sl].mean(0))
                say("%s rules, %s-turn dominant: w %s alpha %s" % (rules, mix, np.round(res[rules, mix][0], 3),
                                                                   np.round(res[rules, mix][1], 3)))
        for mix in ("single", "multi"):
            w = res["algorithms", mix][0]
            assert w[SYS] > w[USER] > max(w[TOOL], w[RESP]) and min(w[TOOL], w[RESP]) > w[COT], (mix, w)
        a = res["algorithms", "multi"][1]
        assert a[CHAT] > a[STRUCT], a
        a = res["algorithms", "single"][1]
        assert a[STRUCT] > a[CHAT], a
        a = res["text", "multi"][1]
        assert a[CHAT] > 4 * a[STRUCT] and a[AGENT] > 4 * a[STRUCT], a
        a = res["text", "single"][1]
        assert a[STRUCT] > a[CHAT] and a[STRUCT] > a[AGENT], a
        w = res["text", "multi"][0]
        assert w[SYS] > max(w[USER], w[TOOL], w[RESP], w[COT]), w
    finally:
        dev.close()
