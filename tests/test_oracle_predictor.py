"""Pins of the session-predictor oracle (Sec. 3.3): the bf16 decoding,
closed forms, a pure-Python brute force on tiny sizes, and the fp32 error
bound (which a float32 evaluation in another order satisfies, and which
planted mistakes exceed)."""
import math

import numpy as np
import pytest

from oracle import predictor as P
from synth import predictor as S

# parity tolerance of the predictor's logit, relative to 1 + |y|: the rigorous fp32
# bound is far too loose here, so the tests below pin this one instead
TOL = 1e-5


def test_bf16_decoding_and_rounding():
    bits = np.array([0x3F80, 0xC000, 0x0000, 0x8000, 0x7F80, 0x3F81, 0x0001, 0x7F7F], np.uint16)
    v = P.bf16_to_f64(bits)
    assert v[0] == 1.0 and v[1] == -2.0 and v[2] == 0.0 and math.copysign(1, v[3]) < 0
    assert v[4] == math.inf and v[5] == 1.0 + 2.0 ** -7 and v[6] == 2.0 ** -133
    assert v[7] == (2.0 - 2.0 ** -7) * 2.0 ** 127
    # round to nearest even: 1 + 2^-8 is a tie (to 1.0), 1 + 3 * 2^-8 rounds up to 1 + 2^-6
    x = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -1.5, 1.0 + 2.0 ** -7 + 2.0 ** -8], np.float32)
    assert S.to_bf16_bits(x).tolist() == [0x3F80, 0x3F82, 0xBFC0, 0x3F82]


def net(d, rng):
    w = S.weights(d, int(rng.integers(1 << 30)))
    h = S.hidden_states(5, d, int(rng.integers(1 << 30)))
    return h, w


def test_closed_form():
    """W1 picks one input per unit, W2 sums pairs, W3 alternates signs."""
    d = 64
    h = S.to_bf16_bits(np.linspace(-3, 3, d, dtype=np.float32)[None, :])
    w1 = np.zeros((256, d), np.float32)
    w1[np.arange(256), np.arange(256) % d] = 1.0
    w2 = np.zeros((64, 256), np.float32)
    w2[np.arange(64), 2 * np.arange(64)] = 1.0
    w2[np.arange(64), 2 * np.arange(64) + 1] = 1.0
    w3 = np.array([1.0, -1.0] * 32, np.float32)
    y, h1, h2 = P.forward(h, S.to_bf16_bits(w1), np.zeros(256), w2, np.full(64, 0.5), w3, np.array([2.0]))
    x = P.bf16_to_f64(h)[0]
    u = np.maximum(x[np.arange(256) % d], 0)
    v = np.maximum(u[0:128:2] + u[1:128:2] + 0.5, 0)
    assert np.allclose(h1[0], u) and np.allclose(h2[0], v)
    assert y[0] == pytest.approx(float(np.sum(v[0::2]) - np.sum(v[1::2]) + 2.0), abs=1e-12)


def test_brute_force_tiny():
    rng = np.random.default_rng(1)
    d = 64
    h, w = net(d, rng)
    y, _, _ = P.forward(h, w["w1"], w["b1"], w["w2"], w["b2"], w["w3"], w["b3"])
    x = P.bf16_to_f64(h)
    W1 = P.bf16_to_f64(w["w1"])
    for r in range(len(h)):
        a = [max(sum(float(W1[j, i]) * float(x[r, i]) for i in range(d)) + float(w["b1"][j]), 0.0) for j in range(256)]
        b = [max(sum(float(w["w2"][k, j]) * a[j] for j in range(256)) + float(w["b2"][k]), 0.0) for k in range(64)]
        yy = sum(float(w["w3"][k]) * b[k] for k in range(64)) + float(w["b3"][0])
        assert y[r] == pytest.approx(yy, rel=1e-12, abs=1e-12)


def test_error_bound_holds_and_catches_mistakes():
    rng = np.random.default_rng(2)
    d = 4096
    h, w = net(d, rng)
    y, _, _ = P.forward(h, w["w1"], w["b1"], w["w2"], w["b2"], w["w3"], w["b3"])
    eb = P.error_bound(h, w["w1"], w["b1"], w["w2"], w["b2"], w["w3"], w["b3"])
    # a float32 evaluation, summed in numpy's own (blocked) order
    x32 = P.bf16_to_f64(h).astype(np.float32)
    W132 = P.bf16_to_f64(w["w1"]).astype(np.float32)
    a = np.maximum(x32 @ W132.T + w["b1"], np.float32(0))
    b = np.maximum(a @ w["w2"].T + w["b2"], np.float32(0))
    y32 = b @ w["w3"] + w["b3"][0]
    assert np.all(np.abs(y32 - y) <= eb), (np.abs(y32 - y), eb)
    # the worst-case bound is loose (sums of absolute terms); the parity
    # tolerance TOL (1 + |y|) holds with a tenfold margin for fp32 evaluations
    # in blocked and in plain sequential order (the sequential one, the worst,
    # stays below 1e-6 here), and planted mistakes land far outside it
    tol = TOL * (1 + np.abs(y))
    assert np.all(np.abs(y32 - y) <= tol / 10)
    h1s = x32[:, 0:1] * W132[:, 0][None, :]
    for i in range(1, d):
        h1s = h1s + x32[:, i:i + 1] * W132[:, i][None, :]
    a2 = np.maximum(h1s + w["b1"], np.float32(0))
    b2 = a2[:, 0:1] * w["w2"][:, 0][None, :]
    for j in range(1, 256):
        b2 = b2 + a2[:, j:j + 1] * w["w2"][:, j][None, :]
    b2 = np.maximum(b2 + w["b2"], np.float32(0))
    y2 = b2[:, 0] * w["w3"][0]
    for k in range(1, 64):
        y2 = y2 + b2[:, k] * w["w3"][k]
    y2 = y2 + w["b3"][0]
    assert np.all(np.abs(y2 - y) <= tol / 10)
    y_nob2, _, _ = P.forward(h, w["w1"], w["b1"], w["w2"], np.zeros(64), w["w3"], w["b3"])
    y_norelu = (P.bf16_to_f64(h) @ P.bf16_to_f64(w["w1"]).T + w["b1"]) @ w["w2"].T.astype(np.float64)
    y_norelu = np.maximum(y_norelu + w["b2"], 0) @ w["w3"] + w["b3"][0]
    w1x = w["w1"].copy()
    w1x[:, 1:] = w1x[:, :-1]                                    # one input column off
    y_shift, _, _ = P.forward(h, w1x, w["b1"], w["w2"], w["b2"], w["w3"], w["b3"])
    for bad in (y_nob2, y_norelu, y_shift):
        assert np.any(np.abs(bad - y) > 10 * tol)   # a parity check over these rows fails
