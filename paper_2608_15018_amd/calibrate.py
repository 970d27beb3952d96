"""Verification cost model on this GPU: t_verify = t0 + T_exp * |U|.

The paper's routing-aware expansion (Sec. "Routing-aware Adaptive Speculative
Expansion", Eq. of the marginal verification cost) prices each newly
activated expert at T_exp, a latency obtained by runtime measurement or
offline profiling, and checks the model against measured verification
latency with R^2 and MAPE.  This module measures the verify-MoE layer pass
over sweeps of draft-batch size B, bias alpha and input seed -- each run
activates some |U| experts -- and fits t0 and T_exp by least squares.

    python -m paper_2608_15018_amd.calibrate --workload c2 [--out file.json]

Timing: per configuration, `steps` back-to-back passes between one pair of
HIP events on the launch stream, cycling through copies of the expert
weights large enough that the last-level cache cannot serve a pass from the
previous one (the protocol of bench.py); the average is used.  Two
latencies are fitted: the whole pass (one s2moe_moe_layer call: route ->
gate -> experts -> combine) and the expert-FFN call alone.
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


# Timed passes cycle through copies of the expert weights that together
# exceed this many bytes, so that the 256 MB last-level cache cannot serve a
# pass from the previous one (the protocol of bench.py).
ROTATE_BYTES = 600_000_000


def expert_bytes(shape, F: int) -> int:
    """HBM bytes of one expert's gate, up and down weights (int4 scales included)."""
    n = 3 * F * shape.hidden
    if shape.wdt == "bf16":
        return 2 * n
    if shape.wdt == "f32":
        return 4 * n
    return n // 2 + 2 * (n // 32)


def sample_inputs(wl, shape, B: int, seed: int, reject_for=None):
    """Router, hidden states and confidences of one sample.  `reject_for`,
    if given, maps the router to a synth.gen.make_batch rejection callback
    (tokens to redraw), e.g. one that keeps every ranking decision clear of
    ties."""
    from synth import gen  # the repository root is on sys.path (run from there)
    from synth.configs import WORKLOAD_ID

    wid = WORKLOAD_ID[wl.name]
    router = gen.make_router(shape, seed, 0, wid, wl.router_std)
    reject = reject_for(router) if reject_for is not None else None
    x, conf_w, _ = gen.make_batch(shape, B, seed, 0, wid, wl.rho, reject)
    return router, x, conf_w


def measure(workload: str, batches, alphas, seeds, steps: int = 20, device="cuda",
            shape=None, reject_for=None, rotate_bytes: int = ROTATE_BYTES) -> list:
    """One sample per (B, alpha, seed): |U| and the average latency (us) of a
    whole pass (route -> gate -> experts -> combine) and of the expert-FFN
    call alone.  Each latency is `steps` back-to-back passes between one pair
    of HIP events on the launch stream, cycling through copies of the expert
    weights (at least `rotate_bytes` of activated weights per cycle, at most
    16 copies), after a short GPU spin that keeps the host ahead.  `shape`
    overrides the workload's layer shape (same generator); `reject_for(router,
    shape)` may supply a make_batch rejection callback per sample."""
    import math

    import torch

    from . import _lib
    from .pipeline import VerifyPass, pack_expert_weights, to_device, weights_to_device
    from synth import gen
    from synth.configs import WORKLOAD_ID, WORKLOADS

    wl = WORKLOADS[workload]
    shape0 = shape or wl.shape
    wid = WORKLOAD_ID[wl.name]
    stream = torch.cuda.current_stream()
    samples = []
    for seed in seeds:
        experts = gen.make_experts(shape0, seed, 0, wid, wl.w_std)
        shared = gen.make_shared_experts(shape0, seed, 0, wid, wl.w_std)
        dev_w, _ = weights_to_device(experts, shared, device)
        packed = shape0.wdt != "f32"
        if packed:
            dev_w, wstruct = pack_expert_weights(dev_w, shape0.wdt)
        else:
            wstruct = _lib.make_weights(*dev_w)
        del experts, shared
        copies = [(wstruct, None)]
        for B in batches:
            for alpha in alphas:
                shape = shape0.with_(alpha=alpha)
                rf = (lambda r, sh=shape: reject_for(r, sh)) if reject_for is not None else None
                router, x, conf_w = sample_inputs(wl, shape, B, seed, rf)
                rd, xd, cd = (to_device(a, device) for a in (router, x, conf_w))
                layer = _lib.make_layer(shape, flags=shape.flags | (
                    _lib.PACKED_WEIGHTS if packed else 0))
                p = VerifyPass(layer, B, device, fused=True)
                p(xd, rd, cd, wstruct)
                torch.cuda.synchronize()
                n_uniq = int(p.rt.n_uniq.item())
                nbytes = (n_uniq * expert_bytes(shape, shape.ffn) +
                          shape.n_shared * expert_bytes(shape, shape.ffn_shared))
                want = max(1, min(16, math.ceil(rotate_bytes / max(1, nbytes))))
                while len(copies) < want:
                    ce = {n: t.clone() for n, t in dev_w[0].items()}
                    cs = {n: t.clone() for n, t in dev_w[1].items()}
                    copies.append((_lib.make_weights(ce, cs), (ce, cs)))
                ws = [c[0] for c in copies[:want]]
                for w in ws:
                    p(xd, rd, cd, w)
                torch.cuda.synchronize()
                t = {}
                for kind in ("step", "ffn"):
                    e0 = torch.cuda.Event(enable_timing=True)
                    e1 = torch.cuda.Event(enable_timing=True)
                    torch.cuda._sleep(2_000_000)
                    e0.record(stream)
                    for i in range(steps):
                        if kind == "step":
                            p(xd, rd, cd, ws[i % want])
                        else:
                            p.verify_moe(xd, ws[i % want])
                    e1.record(stream)
                    torch.cuda.synchronize()
                    t[kind] = e0.elapsed_time(e1) * 1e3 / steps
                samples.append({"B": B, "alpha": alpha, "seed": seed, "n_uniq": n_uniq,
                                "n_shared": shape.n_shared, "weight_copies": want,
                                "t_step_us": t["step"], "t_ffn_us": t["ffn"]})
                print(json.dumps(samples[-1]), file=sys.stderr, flush=True)
        del dev_w, wstruct, copies
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
