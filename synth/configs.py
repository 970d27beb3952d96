"""The synthetic MoE-layer workloads used for parity tests and measurement.

Expert counts, top-k and cap values follow the paper's model table
(Table "Model and SD configurations"): 128 experts top-8 with cap 14 is the
Qwen3 row, 64 experts top-6 with cap 16 is the DeepSeek row.  The paper's
advice to keep cap between 1.5x and 2.5x top-k (Sec. Hyperparameter
Sensitivity, "Effect of reuse-aware gating cap") sets cap = 2k for the
Mixtral-shaped layers.  Draft-tree sizes follow the paper's draft length 8 and
width 2 (Sec. System Implementation, "Draft configuration").
"""

from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class LayerShape:
    """Shape and hyper-parameters of one MoE layer (mirrors ``s2moe_layer``)."""

    hidden: int          # H, model width (K of gate/up, rows of down)
    ffn: int             # F, routed-expert SwiGLU width
    n_experts: int       # E, routed experts
    top_k: int           # k, experts per token
    n_shared: int = 0    # S, always-on shared experts
    ffn_shared: int = 0  # F_s, shared-expert SwiGLU width
    cap: int = 0         # |E*| bound of the globally preferred set
    alpha: float = 0.5   # lambda_b = alpha * gap_b
    flags: int = 0
    act: str = "bf16"    # dtype of x and router: "f32" | "bf16"
    wdt: str = "bf16"    # dtype of expert weights: "f32" | "bf16" | "q4g32"

    def with_(self, **kw) -> "LayerShape":
        d = dict(self.__dict__)
        d.update(kw)
        return LayerShape(**d)


@dataclass(frozen=True)
class Workload:
    name: str
    shape: LayerShape
    batches: tuple            # draft-token counts B this workload is run at
    rho: float                # cross-token correlation of the hidden states
    router_std: float | None  # None -> 1/sqrt(H) (router logits ~ unit variance)
    w_std: float = 0.02       # expert weight std (and fp32 router std for c1)
    n_layers: int = 1
    alphas: tuple = field(default_factory=tuple)  # swept alpha values
    description: str = ""


WORKLOADS = {
    "c1": Workload(
        name="c1",
        shape=LayerShape(hidden=256, ffn=512, n_experts=8, top_k=2, cap=4,
                         alpha=0.5, act="f32", wdt="f32"),
        batches=(8,), rho=0.0, router_std=0.02,
        description="tiny fp32 layer: H 256, F 512, 8 experts top-2, 8 draft tokens",
    ),
    "c2": Workload(
        name="c2",
        shape=LayerShape(hidden=4096, ffn=14336, n_experts=8, top_k=2, cap=4,
                         alpha=0.5, act="bf16", wdt="bf16"),
        batches=(16,), rho=0.6, router_std=None,
        description="Mixtral-8x7B-shaped bf16 layer: H 4096, F 14336, 8 experts "
                    "top-2, 16 draft tokens",
    ),
    "c3": Workload(
        name="c3",
        shape=LayerShape(hidden=2048, ffn=768, n_experts=128, top_k=8, cap=14,
                         alpha=0.5, act="bf16", wdt="bf16"),
        batches=(32,), rho=0.5, router_std=None, alphas=(0.0, 0.5, 1.0),
        description="fine-grained bf16 layer: H 2048, F 768, 128 experts top-8, "
                    "32 draft tokens, alpha swept {0, 0.5, 1}",
    ),
    "c4": Workload(
        name="c4",
        shape=LayerShape(hidden=2048, ffn=1408, n_experts=64, top_k=6, n_shared=2,
                         ffn_shared=1408, cap=16, alpha=0.5, act="bf16",
                         wdt="bf16"),
        batches=(64,), rho=0.4, router_std=None,
        description="shared+routed bf16 layer: H 2048, 2 shared + 64 routed "
                    "experts of F 1408, top-6, 64 draft tokens",
    ),
    "c5": Workload(
        name="c5",
        shape=LayerShape(hidden=4096, ffn=14336, n_experts=8, top_k=2, cap=4,
                         alpha=0.5, act="bf16", wdt="q4g32"),
        batches=(1, 4, 16, 64), rho=0.6, router_std=None, n_layers=24,
        description="24 Mixtral-shaped layers, int4 weights in 32-wide groups "
                    "with fp16 scales, draft sizes {1, 4, 16, 64}",
    ),
}

# A stable small integer per workload name for seed derivation.
WORKLOAD_ID = {name: i + 1 for i, name in enumerate(sorted(WORKLOADS))}


def get_workload(name: str) -> Workload:
    try:
        return WORKLOADS[name]
    except KeyError:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(WORKLOADS)}")
