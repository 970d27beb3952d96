"""Verification cost model on this GPU: t_verify = t0 + T_exp * |U|.

The paper's routing-aware expansion (Sec. "Routing-aware Adaptive Speculative
Expansion", Eq. of the marginal verification cost) prices each newly
activated expert at T_exp, a latency obtained by runtime measurement or
offline profiling, and checks the model against measured verification
latency with R^2 and MAPE.  This module measures the verify-MoE layer pass
over sweeps of draft-batch size B, bias alpha and input seed -- each run
activates some |U| experts -- and fits t0 and T_exp by least squares.

    python -m paper_2608_15018_amd.calibrate --workload c2 [--out file.json]

Timing: per configuration, `steps` passes after one warm-up pass, each
timed with HIP events on the launch stream after a 512 MiB write that
evicts the caches; the median is used.  Two latencies are fitted: the whole
pass (route -> gate -> experts -> combine) and the expert-FFN call alone.
"""

from __future__ import annotations

import argparse
import json
import sys

import numpy as np


def fit_linear(u, t) -> dict:
    """Least-squares t = t0 + T_exp * u with R^2 and MAPE (in %)."""
    u = np.asarray(u, dtype=np.float64)
    t = np.asarray(t, dtype=np.float64)
    if u.size < 2 or np.ptp(u) == 0:
        raise ValueError("need at least two distinct expert counts")
    A = np.stack([np.ones_like(u), u], axis=1)
    (t0, t_exp), *_ = np.linalg.lstsq(A, t, rcond=None)
    pred = t0 + t_exp * u
    ss_res = float(np.sum((t - pred) ** 2))
    ss_tot = float(np.sum((t - t.mean()) ** 2))
    r2 = 1.0 - ss_res / ss_tot if ss_tot > 0 else 1.0
    mape = float(np.mean(np.abs((t - pred) / t))) * 100.0
    return {"t0_us": float(t0), "T_exp_us": float(t_exp), "r2": r2, "mape_pct": mape,
            "n": int(u.size)}


def measure(workload: str, batches, alphas, seeds, steps: int = 20, device="cuda") -> list:
    """One sample per (B, alpha, seed): |U| and median step / FFN latency (us)."""
    import torch

    from . import _lib
    from .pipeline import VerifyPass, pack_expert_weights, to_device, weights_to_device
    from synth import gen  # the repository root is on sys.path (run from there)
    from synth.configs import WORKLOAD_ID, WORKLOADS

    wl = WORKLOADS[workload]
    wid = WORKLOAD_ID[wl.name]
    scrub = torch.empty(512 << 20, dtype=torch.uint8, device=device)
    stream = torch.cuda.current_stream()
    samples = []
    for seed in seeds:
        router = to_device(gen.make_router(wl.shape, seed, 0, wid, wl.router_std), device)
        experts = gen.make_experts(wl.shape, seed, 0, wid, wl.w_std)
        shared = gen.make_shared_experts(wl.shape, seed, 0, wid, wl.w_std)
        dev_w, _ = weights_to_device(experts, shared, device)
        packed = wl.shape.wdt != "f32"
        if packed:
            dev_w, wstruct = pack_expert_weights(dev_w, wl.shape.wdt)
        else:
            wstruct = _lib.make_weights(*dev_w)
        del experts, shared
        for B in batches:
            x, conf_w, _ = gen.make_batch(wl.shape, B, seed, 0, wid, wl.rho)
            xd, cd = to_device(x, device), to_device(conf_w, device)
            for alpha in alphas:
                shape = wl.shape.with_(alpha=alpha)
                layer = _lib.make_layer(shape, flags=shape.flags | (
                    _lib.PACKED_WEIGHTS if packed else 0))
                p = VerifyPass(layer, B, device)
                p(xd, router, cd, wstruct)
                torch.cuda.synchronize()
                n_uniq = int(p.rt.n_uniq.item())
                t_step, t_ffn = [], []
                for i in range(steps):
                    e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
                    scrub.fill_(i & 0xFF)
                    e[0].record(stream)
                    p.route(xd, router)
                    p.reuse_gate(cd)
                    e[1].record(stream)
                    p.verify_moe(xd, wstruct)
                    e[2].record(stream)
                    p.combine()
                    e[3].record(stream)
                    torch.cuda.synchronize()
                    t_step.append(e[0].elapsed_time(e[3]) * 1e3)
                    t_ffn.append(e[1].elapsed_time(e[2]) * 1e3)
                samples.append({"B": B, "alpha": alpha, "seed": seed, "n_uniq": n_uniq,
                                "n_shared": shape.n_shared,
                                "t_step_us": float(np.median(t_step)),
                                "t_ffn_us": float(np.median(t_ffn))})
                print(json.dumps(samples[-1]), file=sys.stderr, flush=True)
        del dev_w, wstruct
        torch.cuda.empty_cache()
    return samples


def calibrate(samples: list) -> dict:
    u = [s["n_uniq"] for s in samples]
    return {"step": fit_linear(u, [s["t_step_us"] for s in samples]),
            "ffn": fit_linear(u, [s["t_ffn_us"] for s in samples])}


SWEEPS = {
    # B spans the draft-batch sizes of each workload family; alpha the bias
    # strengths the paper sweeps; seeds vary the routing.
    "c2": {"batches": [1, 2, 4, 8, 16, 32], "alphas": [0.0, 0.5, 1.0], "seeds": [1, 2]},
    "c3": {"batches": [2, 4, 8, 16, 32, 64], "alphas": [0.0, 0.5, 1.0], "seeds": [1, 2]},
    "c4": {"batches": [2, 4, 8, 16, 32, 64], "alphas": [0.0, 0.5, 1.0], "seeds": [1]},
    "c5": {"batches": [1, 4, 16, 64], "alphas": [0.0, 0.5, 1.0], "seeds": [1, 2]},
}


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--workload", default="c2", choices=sorted(SWEEPS))
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--out", default=None, help="write samples and fit as JSON here")
    args = ap.parse_args(argv)
    from . import _lib
    _lib.load()
    sw = SWEEPS[args.workload]
    samples = measure(args.workload, sw["batches"], sw["alphas"], sw["seeds"], args.steps)
    fit = calibrate(samples)
    result = {"workload": args.workload, "fit": fit, "samples": samples}
    if args.out:
        with open(args.out, "w") as f:
            json.dump(result, f, indent=1)
    print(json.dumps({"workload": args.workload, "fit": fit}))
    return 0


if __name__ == "__main__":
    sys.exit(main())
