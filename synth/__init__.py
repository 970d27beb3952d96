"""Seeded synthetic inputs for the verify-MoE pass and the draft-tree
expansion that selects its tokens.

This package only draws random numbers and stores them in the input formats
(fp32, bf16 bit patterns, packed 4-bit codes with fp16 group scales).  It does
none of the method's arithmetic: routing, gating, the expert FFN and the
combine live in the HIP library and, separately, in the fp64 oracle.  Both
sides read the arrays produced here.
"""

from .configs import WORKLOADS, LayerShape, Workload, get_workload  # noqa: F401
from .gen import (  # noqa: F401
    bf16_bits_from_f32,
    draft_tree_confidence,
    make_batch,
    make_experts,
    make_router,
    make_shared_experts,
)
from .trees import TREE_WORKLOADS, TreeWorkload, make_tree, make_trees  # noqa: F401
