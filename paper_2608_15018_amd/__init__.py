"""S2-MoE verify-MoE hot path for AMD Instinct MI355X (gfx950), and the
routing-aware draft-tree expansion that selects its tokens.

The work happens in libs2moe.so (hand-written HIP, C ABI in include/s2moe.h);
this package is its thin Python binding.
"""

from ._lib import (  # noqa: F401
    BF16,
    BIAS_ABSOLUTE,
    ExpandOut,
    F32,
    GATE_FROM_BIASED,
    PACKED_WEIGHTS,
    PREF_ACTIVATED_ONLY,
    Q4G32,
    Layer,
    NOALLOC_SCRATCH_BYTES,
    Routing,
    STREAM_SINK_WORDS,
    S2moeError,
    Weights,
    abi_version,
    combine,
    expand,
    expand_max_nodes,
    load,
    make_layer,
    make_weights,
    moe_layer,
    pack_weights,
    reuse_gate,
    route,
    stream_read,
    verify_moe,
    verify_moe_noalloc,
    workspace_bytes,
)
from .pipeline import (  # noqa: F401
    VerifyPass,
    pack_expert_weights,
    to_device,
    weights_to_device,
)
