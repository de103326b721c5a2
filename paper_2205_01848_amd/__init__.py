"""MI355X (gfx950) MoE layer with dynamic per-expert capacities and cached
assignments: libmoe.so (HIP kernels behind a C ABI, include/moe.h) and its
thin Python binding."""
from . import binding  # noqa: F401
from .layer import MoELayer, rows_alloc_for  # noqa: F401

__all__ = ["binding", "MoELayer", "rows_alloc_for"]
