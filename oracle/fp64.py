"""TEST INFRASTRUCTURE — Eq. 1-3 in fp64 with the C library's log/erfc/pow.

This is the accuracy reference the fp32 recipe (oracle/dsr.c) is pinned to;
it is never used to take a selection decision.
"""
import math


def p_lognormal(dt, mu, sigma):
    """Eq. 1: 1 - F_LN(dt; mu, sigma) = erfc((ln dt - mu) / (sigma sqrt 2)) / 2."""
    return 0.5 * math.erfc((math.log(dt) - mu) / (sigma * math.sqrt(2.0)))


def p_structural(ob, omax, gamma):
    """Eq. 2: 1 - (o_b / o_max)^gamma, with o_max = 0 read as the first block."""
    r = 0.0 if omax == 0 else min(ob / omax, 1.0)
    return 1.0 - r ** gamma


def priority(alpha, w, p, dt):
    """Eq. 3: P = alpha_q w_tau p / dt, +inf at dt = 0."""
    return math.inf if dt == 0 else alpha * w * p / dt
