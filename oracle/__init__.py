"""CPU oracle of the capacity-bounded top-k MoE layer.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package; the product path
(the HIP library and its Python binding) never does.  It shares no code with
the HIP path: plain numpy in float64, one step per function, each citing the
passage of the paper (Kossmann, Jia, Aiken, "Optimizing Mixture of Experts
using Dynamic Recompilations", MLSys 2022) that it follows.
"""
from .moe_oracle import *  # noqa: F401,F403
from .moe_oracle import __all__  # noqa: F401
