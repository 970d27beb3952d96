"""Seeded synthetic expert weights generated directly in device memory.

For benchmark stacks too large to draw on the host (tens of GB).  Draws
only: N(0, std^2) bf16 weights, or uniform 4-bit codes with fp16 group
scales s = std / 4.61 * (1 +- 25 % uniform jitter), with the same formats
and shapes as `synth.gen` (gate/up [n, F, H], down [n, H, F]).  Values come
from torch's generator on the device, seeded per (seed, layer, tensor), so
they differ from `synth.gen`'s host streams; the parity tests use the host
generator.
"""

from __future__ import annotations

import torch


def _gen(device, seed: int, layer: int, tensor: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed((seed * 1_000_003 + layer * 10_007 + tensor) & 0x7FFFFFFFFFFFFFFF)
    return g


def _bf16(shape, std, g, device):
    return (torch.randn(shape, generator=g, device=device, dtype=torch.float32) * std).to(
        torch.bfloat16)


def _q4(shape, std, g, device):
    n, rows, K = shape
    codes = torch.randint(0, 256, (n, rows, K // 2), generator=g, device=device,
                          dtype=torch.int32).to(torch.uint8)
    jitter = torch.rand((n, rows, K // 32), generator=g, device=device) * 0.5 + 0.75
    scales = (jitter * (std / 4.61)).to(torch.float16)
    return codes, scales


def expert_weights(n: int, F: int, H: int, wdt: str, seed: int, layer: int, tag: int = 0,
                   std: float = 0.02, device="cuda") -> dict:
    """{gate, up, down (+ _s scales)} for n experts of width F."""
    out = {}
    for t, (name, shape) in enumerate((("gate", (n, F, H)), ("up", (n, F, H)),
                                       ("down", (n, H, F)))):
        g = _gen(device, seed, layer, 16 * tag + t)
        if wdt == "bf16":
            out[name] = _bf16(shape, std, g, device)
        elif wdt == "q4g32":
            out[name], out[name + "_s"] = _q4(shape, std, g, device)
        else:
            raise ValueError(f"unsupported weight dtype {wdt}")
    return out


def activations(B: int, H: int, seed: int, layer: int, rho: float, device="cuda"):
    """x_b = sqrt(rho) u + sqrt(1 - rho) n_b (bf16) and a router
    W_r ~ N(0, 1/H) for E experts is drawn by `router`."""
    g = _gen(device, seed, layer, 101)
    u = torch.randn(H, generator=g, device=device)
    nz = torch.randn((B, H), generator=g, device=device)
    return ((rho ** 0.5) * u[None] + ((1 - rho) ** 0.5) * nz).to(torch.bfloat16)


def router(E: int, H: int, seed: int, layer: int, device="cuda"):
    g = _gen(device, seed, layer, 102)
    return (torch.randn((E, H), generator=g, device=device) / H ** 0.5).to(torch.bfloat16)
