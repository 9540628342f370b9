"""Trace-replay set-up shared by the oracle side and the HIP side: the paper's
four queues and their starting timing parameters, and the seeded request
generator of every cache instance.  Holds no step of the eviction method and
imports neither the oracle nor the HIP package."""
from synth.pools import MU_AGENT_MS, MU_CHAT_MS, SIGMA_AGENT, SIGMA_CHAT
from synth.trace import TRACE_CONFIGS, TraceGen

# the paper's four queues (Sec. 3.1): evict-first, structural, chat, agent
# (queue kinds: 0 evict-first, 1 structural, 2 log-normal)
KINDS = [0, 1, 2, 2]
ROLES = [0, 1, 2, 3]
MU = [0.0, 0.0, MU_CHAT_MS, MU_AGENT_MS]
SIGMA = [1.0, 1.0, SIGMA_CHAT, SIGMA_AGENT]


def trace_gen(name, inst, n_inst=None, **over):
    """Request generator of instance `inst` of trace configuration `name`."""
    cfg = TRACE_CONFIGS[name]
    n_inst = cfg["n_inst"] if n_inst is None else n_inst
    if "mixes" in cfg:
        mix = cfg["mixes"][0 if inst < n_inst // 2 else 1]
    else:
        mix = cfg["mix"]
    return TraceGen(mix, cfg["seed"] * 1000 + inst, **over)


def trace_gens(name, n_inst, **over):
    return [trace_gen(name, i, n_inst, **over) for i in range(n_inst)]
