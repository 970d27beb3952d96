"""cap x alpha sensitivity of expert reuse under reuse-aware gating.

The paper measures how much reuse-aware gating lowers the reuse ratio
|U| / (B k) of a verify batch (Sec. Experiments, the expert-reuse table,
"Reuse Improvement" = relative reduction) and how the gating cap trades
reuse against routing freedom (Sec. Hyperparameter Sensitivity Analysis,
"Effect of reuse-aware gating cap": 1.5x to 2.5x the top-k works best).
Its numbers come from real routing traces; this module sweeps cap and
alpha on seeded synthetic routing of the paper's DeepSeek and OLMoE layer
shapes, with every routing decision taken by the library's kernels
(s2moe_route once per batch, s2moe_reuse_gate per (cap, alpha)).

    python -m paper_2608_15018_amd.sensitivity [--out file.json] [--md file.md]

Reported per (cap, alpha), as means over the batches:
  reuse ratio r = |U| / (B k);
  improvement 1 - r / r(alpha = 0), the paper's "Reuse Improvement";
  deviation: the share of a batch's B k expert slots that differ from the
  plain top-k, i.e. how far the bias moves the routing.
"""

from __future__ import annotations

import argparse
import json
import sys

import numpy as np

# Experts, top-k and the paper's cap from its model table (Table "Model and
# SD configurations"); hidden sizes from the public architectures.
SHAPES = {
    "deepseek": dict(hidden=2048, ffn=1408, n_experts=64, top_k=6, paper_cap=16),
    "olmoe": dict(hidden=2048, ffn=1024, n_experts=64, top_k=8, paper_cap=18),
}
ALPHAS = (0.0, 0.25, 0.5, 1.0, 2.0, 4.0)
WL_ID = 40  # seed-key tag of these inputs


def caps_for(k: int, paper_cap: int, n_experts: int) -> list:
    """cap in [k, 3k]: k, 1.5k, 2k, 2.5k, 3k (rounded) and the paper's value."""
    c = {k, int(round(1.5 * k)), 2 * k, int(round(2.5 * k)), 3 * k, paper_cap}
    return sorted(x for x in c if k <= x <= n_experts)


def reuse_ratio(idx: np.ndarray, k: int) -> float:
    """|U| / (B k) of one batch's selected experts idx [B, k]."""
    B = idx.shape[0]
    return len(np.unique(idx)) / float(B * k)


def deviation(idx: np.ndarray, plain_idx: np.ndarray) -> float:
    """Share of the B k (token, slot) selections not in the token's plain top-k."""
    moved = sum(len(set(a.tolist()) - set(b.tolist())) for a, b in zip(idx, plain_idx))
    return moved / float(idx.size)


def improvement(r_plain: float, r_gated: float) -> float:
    """The paper's "Reuse Improvement": relative reduction of the ratio."""
    return (r_plain - r_gated) / r_plain


def layer_shape(name: str, cap: int, alpha: float):
    from synth.configs import LayerShape
    s = SHAPES[name]
    return LayerShape(hidden=s["hidden"], ffn=s["ffn"], n_experts=s["n_experts"],
                      top_k=s["top_k"], cap=cap, alpha=alpha, act="bf16", wdt="bf16")


def gpu_selections(name: str, x, router, conf_w, caps, alphas, device="cuda") -> dict:
    """plain_idx and {(cap, alpha): idx} for one batch, from the library's
    routing and gating kernels."""
    import torch

    from . import _lib
    from .pipeline import to_device

    B = x.shape[0]
    base = _lib.make_layer(layer_shape(name, caps[0], 0.0))
    rt = _lib.Routing(base, B, device)
    xd, rd, cd = to_device(x, device), to_device(router, device), to_device(conf_w, device)
    _lib.route(base, xd, rd, rt)
    out = {}
    for cap in caps:
        for alpha in alphas:
            _lib.reuse_gate(_lib.make_layer(layer_shape(name, cap, alpha)), cd, rt)
            torch.cuda.synchronize()
            out[(cap, alpha)] = rt.idx.cpu().numpy().copy()
    plain = rt.plain_idx.cpu().numpy().copy()
    return {"plain_idx": plain, "idx": out}


def batch_inputs(name: str, B: int, seed: int, rho: float):
    """Router [E, H] and a batch (x [B, H], draft-tree confidences [B])."""
    from synth import gen
    shape = layer_shape(name, SHAPES[name]["paper_cap"], 0.5)
    router = gen.make_router(shape, seed, 0, WL_ID)
    x, conf_w, _ = gen.make_batch(shape, B, seed, 0, WL_ID, rho)
    return x, router, conf_w


def summarize(k: int, samples: list, caps, alphas) -> dict:
    """Means over batches; samples are gpu_selections results."""
    res = {}
    r0 = np.mean([reuse_ratio(s["idx"][(caps[0], 0.0)], k) for s in samples])
    for cap in caps:
        for alpha in alphas:
            r = np.mean([reuse_ratio(s["idx"][(cap, alpha)], k) for s in samples])
            dev = np.mean([deviation(s["idx"][(cap, alpha)], s["plain_idx"]) for s in samples])
            res[f"{cap}/{alpha}"] = {"cap": cap, "alpha": alpha, "reuse_ratio": float(r),
                                    "improvement": float(improvement(r0, r)),
                                    "deviation": float(dev)}
    return {"plain_reuse_ratio": float(r0), "grid": res}


def sweep(name: str, B: int, seeds, rho: float, alphas=ALPHAS) -> dict:
    s = SHAPES[name]
    caps = caps_for(s["top_k"], s["paper_cap"], s["n_experts"])
    samples = []
    for seed in seeds:
        x, router, conf_w = batch_inputs(name, B, seed, rho)
        samples.append(gpu_selections(name, x, router, conf_w, caps, alphas))
    out = summarize(s["top_k"], samples, caps, alphas)
    out.update({"shape": name, "B": B, "rho": rho, "batches": len(samples), "caps": caps,
                "alphas": list(alphas), "k": s["top_k"], "paper_cap": s["paper_cap"]})
    return out


def to_markdown(results: list) -> str:
    lines = []
    for r in results:
        lines += [f"### {r['shape']}: E = 64, k = {r['k']}, paper cap {r['paper_cap']}, "
                  f"B = {r['B']}, rho = {r['rho']}, {r['batches']} batches",
                  "", f"Plain reuse ratio (alpha = 0): {r['plain_reuse_ratio']:.4f}.  Cells: reuse "
                  "ratio / improvement % / deviation %.", "",
                  "| cap | " + " | ".join(f"alpha {a:g}" for a in r["alphas"]) + " |",
                  "|---" * (len(r["alphas"]) + 1) + "|"]
        for cap in r["caps"]:
            cells = []
            for a in r["alphas"]:
                g = r["grid"][f"{cap}/{a}"]
                cells.append(f"{g['reuse_ratio']:.3f} / {100 * g['improvement']:.1f} / "
                             f"{100 * g['deviation']:.1f}")
            tag = f"{cap} ({cap / r['k']:.2g}k)" + (" paper" if cap == r["paper_cap"] else "")
            lines.append(f"| {tag} | " + " | ".join(cells) + " |")
        lines.append("")
    return "\n".join(lines) + "\n"


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--batches", type=int, default=32)
    ap.add_argument("--rho", type=float, default=0.2)
    ap.add_argument("--sizes", default="8,16")
    ap.add_argument("--out", default=None)
    ap.add_argument("--md", default=None)
    args = ap.parse_args(argv)
    results = []
    for name in SHAPES:
        for B in (int(b) for b in args.sizes.split(",")):
            r = sweep(name, B, range(args.batches), args.rho)
            results.append(r)
            print(f"[sensitivity] {name} B={B} plain r={r['plain_reuse_ratio']:.4f}", flush=True)
    if args.out:
        with open(args.out, "w") as f:
            json.dump(results, f, indent=1)
    md = to_markdown(results)
    if args.md:
        with open(args.md, "w") as f:
            f.write(md)
    else:
        sys.stdout.write(md)
    return 0


if __name__ == "__main__":
    sys.exit(main())
