"""TEST INFRASTRUCTURE — CPU oracle of SAECache's eviction hot path.

Plain, slow and independent of the HIP path (no shared code, headers, tables
or constant generators).  Only tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg may import, call, link or execute anything in this package.

  dsr.c      fp32 realisation of Eq. 1-3 (the precision the selection is
             decided in), built with gcc -ffp-contract=off
  fp64.py    Eq. 1-3 in fp64 (accuracy reference for the pins)
  policy.py  selection, Algorithm 1 decision and commit, strict prefix
             matching, Add(), Algorithms 2 and 3, as a per-instance state
             machine
"""
from . import _native, fp64, policy  # noqa: F401
from .policy import (EVICT_FIRST, LOGNORMAL, N_TYPES, RECENCY, STRUCTURAL,  # noqa: F401
                     OracleCache, Params, block_type, classify)


def build():
    """Compile the oracle's C part (gcc)."""
    return _native.build(force=True)
