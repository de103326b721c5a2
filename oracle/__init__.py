"""CPU oracle of the capacity-bounded top-k MoE layer.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package; the product path
(the HIP library and its Python binding) never does.  It shares no code with
the HIP path: plain numpy in float64, one step per function, each citing the
passage of the paper (Kossmann, Jia, Aiken, "Optimizing Mixture of Experts
using Dynamic Recompilations", MLSys 2022) that it follows.
"""
from .moe_oracle import *  # noqa: F401,F403
from .losses import *  # noqa: F401,F403
from .policies import *  # noqa: F401,F403
from . import losses as _losses, moe_oracle as _core, policies as _policies

__all__ = list(_core.__all__) + list(_losses.__all__) + list(_policies.__all__)
