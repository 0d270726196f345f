"""REFLEX variable-K MoE layer for MI355X (gfx950).

The computation lives in ``libreflex.so`` (hand-written HIP kernels behind the C
ABI declared in ``include/reflex.h``).  This package is its Python binding:
``_lib`` mirrors the C entry points one to one, ``layer`` runs the fused layer
from torch tensors.  Importing the package does not load the library; the first
call does, and fails loudly if it has not been built.
"""
from ._lib import (  # noqa: F401
    ReflexError,
    lib,
    reflex_assign_budget,
    reflex_combine,
    reflex_grouped_swiglu,
    reflex_moe_forward,
    reflex_permute,
    reflex_permute_workspace_size,
    reflex_router_logits,
    reflex_swiglu_workspace_size,
    reflex_topk_variable,
    reflex_workspace_size,
)
