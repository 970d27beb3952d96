"""One verify-MoE pass (route -> reuse_gate -> verify_moe -> combine) on one
HIP stream, with the device buffers it needs.  Plumbing only: every step is
a call into libs2moe.so."""

from __future__ import annotations

import numpy as np
import torch

from . import _lib


def to_device(a: np.ndarray, device="cuda") -> torch.Tensor:
    """Host array in a stored format -> device tensor holding the same bytes.
    uint16 arrays are bf16 bit patterns and become torch.bfloat16."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        t = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(a)
    return t.to(device)


def weights_to_device(experts: dict, shared: dict | None, device="cuda"):
    """(device tensors, Weights struct) from host weight dicts."""
    dev_e = {n: to_device(v, device) for n, v in experts.items()}
    dev_s = {n: to_device(v, device) for n, v in (shared or {}).items()}
    return (dev_e, dev_s), _lib.make_weights(dev_e, dev_s)


def pack_expert_weights(dev: tuple, wdt: str):
    """(device tensors, Weights struct) of the packed copies of the device
    weights `dev` = (routed dict, shared dict) from weights_to_device; use
    them with a layer whose flags include PACKED_WEIGHTS."""
    out = []
    for d in dev:
        p = {}
        for n in ("gate", "up", "down"):
            if n in d:
                p[n], sc = _lib.pack_weights(wdt, d[n], d.get(n + "_s"))
                if sc is not None:
                    p[n + "_s"] = sc
        out.append(p)
    return (out[0], out[1]), _lib.make_weights(out[0], out[1])


class VerifyPass:
    """Buffers and calls of one verify-MoE layer pass for B draft tokens.
    With fused=True a call is one s2moe_moe_layer (same results bit for bit,
    fewer launches for small batches); otherwise the four calls in turn."""

    def __init__(self, layer: _lib.Layer, B: int, device="cuda", fused: bool = False):
        self.layer = layer
        self.B = B
        self.fused = fused
        self.rt = _lib.Routing(layer, B, device)
        nbytes = _lib.workspace_bytes(layer, B)
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
        rows = B * layer.top_k + layer.n_shared * B
        self.expert_out = torch.empty((rows, layer.hidden), dtype=torch.float32, device=device)
        self.y = torch.empty((B, layer.hidden), dtype=torch.float32, device=device)

    def route(self, x, router, stream=None):
        _lib.route(self.layer, x, router, self.rt, stream)

    def reuse_gate(self, conf_w, stream=None):
        _lib.reuse_gate(self.layer, conf_w, self.rt, stream)

    def verify_moe(self, x, weights: _lib.Weights, stream=None):
        _lib.verify_moe(self.layer, x, weights, self.rt, self.workspace, self.expert_out, stream)

    def combine(self, stream=None):
        _lib.combine(self.layer, self.rt, self.expert_out, self.y, stream)

    def __call__(self, x, router, conf_w, weights: _lib.Weights, stream=None):
        if self.fused:
            _lib.moe_layer(self.layer, x, router, conf_w, weights, self.rt, self.workspace,
                           self.expert_out, self.y, stream)
            return self.y
        self.route(x, router, stream)
        self.reuse_gate(conf_w, stream)
        self.verify_moe(x, weights, stream)
        self.combine(stream)
        return self.y

    def results(self) -> dict:
        out = self.rt.host()
        out["n_uniq"] = int(out["n_uniq"][0])
        out["expert_out"] = self.expert_out.cpu().numpy()
        out["y"] = self.y.cpu().numpy()
        return out
