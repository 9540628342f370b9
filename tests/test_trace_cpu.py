"""Trace generator and replay driver on the CPU (oracle backend only)."""
import numpy as np

from oracle_backend import OracleBackend
from synth.pools import MU_AGENT_MS, MU_CHAT_MS, SIGMA_AGENT, SIGMA_CHAT
from synth.replay import Replay
from synth.trace import (COT, H_DECODE, H_MULTI_TURN, H_SHARED_PREFIX, H_UNTEMPLATED, MIXES, MULTI_TURN, RESPONSE,
                         SYSTEM, TraceGen)

KINDS, ROLES = [0, 1, 2, 2], [0, 1, 2, 3]
MU, SIGMA = [0.0, 0.0, MU_CHAT_MS, MU_AGENT_MS], [1.0, 1.0, SIGMA_CHAT, SIGMA_AGENT]


def test_trace_is_deterministic():
    a, b = TraceGen("balanced", 7), TraceGen("balanced", 7)
    for _ in range(200):
        x, y = a.next(), b.next()
        assert x["now"] == y["now"] and np.array_equal(x["hashes"], y["hashes"])
        assert np.array_equal(x["hints"], y["hints"]) and np.array_equal(x["types"], y["types"])


def test_request_mix_follows_table2():
    for mix in ("balanced", "multi_turn_dominant", "single_turn_dominant"):
        g = TraceGen(mix, 11)
        cats = np.bincount([g.next()["category"] for _ in range(3000)], minlength=5) / 3000.0
        assert np.all(np.abs(cats - np.array(MIXES[mix])) < 0.03), (mix, cats)


def test_sessions_extend_their_prompts():
    """Turn t+1's prompt starts with turn t's prompt; turn t's response blocks
    follow it (same hashes) exactly when turn t generated no chain-of-thought."""
    g = TraceGen("multi_turn_dominant", 3)
    last = {}
    seen = 0
    for _ in range(3000):
        r = g.next()
        s = r["session"]
        if r["turn"] > 1 and s in last:
            prev = last[s]
            npv = prev["n_prompt"]
            assert np.array_equal(r["hashes"][:npv], prev["hashes"][:npv])
            gen_t = prev["types"][npv:]
            resp = prev["hashes"][npv:][gen_t == RESPONSE]
            nxt = r["hashes"][npv:npv + len(resp)]
            if not (gen_t == COT).any():
                assert np.array_equal(nxt, resp)
            else:
                assert not np.intersect1d(nxt, resp).size
            seen += 1
        last[s] = r
    assert seen > 100


def test_hints_and_types():
    g = TraceGen("balanced", 5)
    for _ in range(1000):
        r = g.next()
        n = r["n_prompt"]
        t, h = r["types"], r["hints"]
        assert not (t[:n] == COT).any()                      # chain-of-thought is generated only
        assert np.all(t[:n][(h[:n] & H_SHARED_PREFIX) != 0] == SYSTEM)
        single = not (h[0] & H_MULTI_TURN) and r["turn"] == 1
        assert np.all(((h[n:] & H_DECODE) != 0) == single)
        assert np.all(((h[:n] & H_UNTEMPLATED) != 0) == (single & ((h[:n] & H_SHARED_PREFIX) == 0)))
        if r["turn"] > 1:
            assert MULTI_TURN[r["category"]] and np.all(h & H_MULTI_TURN)


def test_oracle_replay_accounting():
    """Slots are conserved, referenced blocks are never evicted (the oracle's
    commit asserts it) and every reference is released at the end."""
    cap = 600
    be = OracleBackend([0], cap, KINDS, ROLES, MU, SIGMA, K=32, learn=3)
    rp = Replay(be, 1, cap, k_min=1, max_k=cap, concurrency=4)
    g = TraceGen("balanced", 9, template_tokens=(160, 800))
    for _ in range(400):
        rp.step({0: g.next()})
        c = be.c[0]
        assert c.valid.sum() + len(rp.free[0]) == cap
        assert len(c.index) == c.valid.sum()
    s = rp.summary()
    assert s["evicted"] > 0 and s["hit_blocks"] > 0 and be.c[0].n_updates > 0
    for ids in rp.inflight[0]:
        be.ref(np.zeros(len(ids), np.int32), ids, -1)
    assert (be.c[0].ref_count == 0).all()
