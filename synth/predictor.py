"""Seeded inputs of the session predictor: last-token hidden states of a
d = 4,096 serving model and random-initialised MLP weights (the trained
weights and real hidden states are not available).

* hidden states: N(0, 1) per coordinate, with 8 fixed outlier coordinates of
  scale 20 (final-layer activations of LLMs carry a few large channels),
  rounded to bf16 (round to nearest even);
* W1 ~ N(0, 2 / d) (He initialisation for a ReLU layer) in bf16, W2 ~
  N(0, 2 / 256), W3 ~ N(0, 1 / 64) in fp32, biases N(0, 0.01^2).
"""
import numpy as np

H1, H2 = 256, 64


def to_bf16_bits(x):
    """float32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    r = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return r.astype(np.uint16)


def hidden_states(n, d, seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n, d), dtype=np.float32)
    out = np.random.default_rng(seed ^ 0x5A5A).choice(d, size=min(8, d), replace=False)
    x[:, out] *= 20.0
    return to_bf16_bits(x)


def weights(d, seed):
    rng = np.random.default_rng(seed)
    w1 = to_bf16_bits(rng.standard_normal((H1, d), dtype=np.float32) * np.float32(np.sqrt(2.0 / d)))
    b1 = (rng.standard_normal(H1) * 0.01).astype(np.float32)
    w2 = (rng.standard_normal((H2, H1)) * np.sqrt(2.0 / H1)).astype(np.float32)
    b2 = (rng.standard_normal(H2) * 0.01).astype(np.float32)
    w3 = (rng.standard_normal(H2) * np.sqrt(1.0 / H2)).astype(np.float32)
    b3 = (rng.standard_normal(1) * 0.01).astype(np.float32)
    return dict(w1=w1, b1=b1, w2=w2, b2=b2, w3=w3, b3=b3)
