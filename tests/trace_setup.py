"""Trace-replay set-up shared by the oracle side and the HIP side (re-exported
from synth.trace): the paper's four queues and their starting timing
parameters, and the seeded request generator of every cache instance.  Holds
no step of the eviction method and imports neither the oracle nor the HIP
package."""
from synth.trace import TRACE_KINDS as KINDS  # noqa: F401
from synth.trace import TRACE_MU as MU  # noqa: F401
from synth.trace import TRACE_ROLES as ROLES  # noqa: F401
from synth.trace import TRACE_SIGMA as SIGMA  # noqa: F401
from synth.trace import trace_gen, trace_gens  # noqa: F401
