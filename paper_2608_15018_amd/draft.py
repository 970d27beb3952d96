"""Expert-sparse self-draft pass on the verify-MoE kernels.

The paper drafts with the target model itself, run with fewer experts per
token (Sec. System Implementation, "Draft configuration"; the "Draft
Experts" column of its model table): k_draft = 2 for OLMoE, 1 for DeepSeek
and GPT-OSS, 3 for Qwen3, optionally quantised.  A draft step therefore
runs every MoE layer at its smallest shape: B = 1 (or the few tokens of one
draft-tree level), top-k_draft routing without reuse bias (alpha = 0), the
k_draft experts' FFN and the combine -- the same library calls as
verification.  Attention and the rest of the transformer are out of scope:
each layer takes its own hidden states.

At these shapes a layer streams a few MB of weights, so launch latency
matters: each layer is one s2moe_moe_layer call (three launches instead of
six where the batch allows, the same results bit for bit), and a
`DraftStep` can be captured once in a HIP graph (through torch's graph
capture of the stream the library calls enqueue on) and replayed.
"""

from __future__ import annotations

import torch

from . import _lib
from .pipeline import VerifyPass

# Hidden size, expert width, experts, top-k, MoE layers and shared experts
# from the public architectures; k_draft from the paper's model table.
DRAFT_MODELS = {
    "olmoe": dict(hidden=2048, ffn=1024, n_experts=64, top_k=8, k_draft=2, layers=16),
    "deepseek": dict(hidden=2048, ffn=1408, n_experts=64, top_k=6, k_draft=1, layers=26,
                     n_shared=2, ffn_shared=1408),
    "qwen3": dict(hidden=2048, ffn=768, n_experts=128, top_k=8, k_draft=3, layers=48),
    "gptoss": dict(hidden=2880, ffn=2880, n_experts=128, top_k=4, k_draft=1, layers=36),
}


def draft_layer(model: str, wdt: str = "bf16", k_draft: int | None = None, packed=True):
    """Layer struct of the draft pass: top-k_draft, no reuse bias (alpha 0,
    cap = k_draft), bf16 activations."""
    m = DRAFT_MODELS[model]
    k = m["k_draft"] if k_draft is None else k_draft
    return _lib.make_layer(hidden=m["hidden"], ffn=m["ffn"], n_experts=m["n_experts"], top_k=k,
                           n_shared=m.get("n_shared", 0), ffn_shared=m.get("ffn_shared", 0),
                           cap=k, alpha=0.0, act="bf16", wdt=wdt,
                           flags=_lib.PACKED_WEIGHTS if packed else 0)


class DraftStep:
    """One draft step over a stack of layers: for layer l, route ->
    gate -> experts -> combine on inputs (x_l, router_l, weights_l)."""

    def __init__(self, layer: _lib.Layer, B: int, inputs: list, device="cuda",
                 fused: bool = True):
        """inputs: per layer (x [B, H] bf16, router [E, H] bf16, Weights).
        fused=False runs each layer as the four separate calls instead of one
        s2moe_moe_layer."""
        self.layer = layer
        self.B = B
        self.inputs = inputs
        self.conf = torch.ones(B, dtype=torch.float32, device=device)
        self.passes = [VerifyPass(layer, B, device, fused=fused) for _ in inputs]
        self.graph = None

    def __call__(self, stream=None):
        for p, (x, router, w) in zip(self.passes, self.inputs):
            p(x, router, self.conf, w, stream)

    def capture(self):
        """Record one step into a HIP graph (the library issues no memset or
        allocation, so the whole step is capturable)."""
        torch.cuda.synchronize()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            self()  # warm-up on a side stream, as graph capture requires
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            self()
        return self.graph

    def replay(self):
        self.graph.replay()

    def outputs(self) -> list:
        return [p.y for p in self.passes]
