"""fp64 CPU oracle (test infrastructure; see s2moe_oracle)."""

from . import expand_oracle, s2moe_oracle  # noqa: F401
from .s2moe_oracle import (  # noqa: F401
    BIAS_ABSOLUTE,
    GATE_FROM_BIASED,
    PREF_ACTIVATED_ONLY,
    bucket,
    combine,
    dequant_q4g32,
    forward,
    reuse_gate,
    margin_reject,
    reuse_improvement,
    route,
    routing_margins,
    upcast,
    verify_moe,
)
