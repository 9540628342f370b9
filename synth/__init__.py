"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and bench.py.

This module holds none of the eviction method's arithmetic: it only draws
pool features, hash chains and request batches with the shapes and
distributions of the workloads being exercised.  Nothing here scores, sorts,
selects, classifies a block type or learns.

Every draw comes from numpy's PCG64 seeded through SeedSequence(seed), with
one spawned child stream per field, so the same seed gives the same bytes.
"""
from .pools import (CONFIGS, MU_AGENT_MS, MU_CHAT_MS, SIGMA_AGENT, SIGMA_CHAT,  # noqa: F401
                    chain_hashes, make_pool, make_requests, mix64, pool_config)
