"""TEST INFRASTRUCTURE — CPU oracle of the multi-turn session predictor
(Sec. 3.3): y = W3 relu(W2 relu(W1 h + b1) + b2) + b3, hidden widths 256 and
64, y > 0 predicting that the session continues.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may use
it.  Plain fp64 with numpy matrix products on the exact values of the bf16
and fp32 inputs, plus the rounding-error bound that any fp32 evaluation of
the same formula (any summation order, exact bf16 products) satisfies.
"""
import numpy as np

U = 2.0 ** -24  # unit roundoff of fp32


def bf16_to_f64(bits):
    """bf16 bit patterns (uint16) -> their exact values: the upper half of an
    IEEE binary32."""
    b = np.asarray(bits, np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def forward(h_bits, w1_bits, b1, w2, b2, w3, b3):
    """Returns (y, h1, h2) in fp64 for every row of h."""
    h = bf16_to_f64(h_bits)
    W1 = bf16_to_f64(w1_bits)
    h1 = np.maximum(h @ W1.T + np.asarray(b1, np.float64), 0.0)
    h2 = np.maximum(h1 @ np.asarray(w2, np.float64).T + np.asarray(b2, np.float64), 0.0)
    y = h2 @ np.asarray(w3, np.float64) + float(np.asarray(b3, np.float64).reshape(-1)[0])
    return y, h1, h2


def gamma(n):
    return n * U / (1.0 - n * U)


def error_bound(h_bits, w1_bits, b1, w2, b2, w3, b3):
    """Per row, a bound on |y_fp32 - y| for an fp32 evaluation in any order:
    each dot product of length m plus its bias is within gamma(m + 1) times
    its sum of absolute terms; ReLU is 1-Lipschitz; the errors of one layer
    propagate through the next layer's absolute weights."""
    h = np.abs(bf16_to_f64(h_bits))
    W1 = np.abs(bf16_to_f64(w1_bits))
    A1 = h @ W1.T + np.abs(np.asarray(b1, np.float64))
    e1 = gamma(h.shape[1] + 1) * A1
    _, h1, h2 = forward(h_bits, w1_bits, b1, w2, b2, w3, b3)
    W2 = np.abs(np.asarray(w2, np.float64))
    A2 = (h1 + e1) @ W2.T + np.abs(np.asarray(b2, np.float64))
    e2 = e1 @ W2.T + gamma(W2.shape[1] + 1) * A2
    W3 = np.abs(np.asarray(w3, np.float64))
    A3 = (h2 + e2) @ W3 + abs(float(np.asarray(b3).reshape(-1)[0]))
    return e2 @ W3 + gamma(W3.shape[0] + 1) * A3
