"""Shared helpers of the GPU parity tests: seeded inputs, one pass through
the C ABI, the oracle on the same inputs, and the comparisons."""

from __future__ import annotations

import sys

import numpy as np

import oracle
from synth import gen

# Tolerances (max |gpu - ref| / max |ref| over the whole array).
TOL_Y = {"f32": 1e-4, "bf16": 2e-2, "q4g32": 2e-2}  # expert_out and y
TOL_ROUTER = 1e-5                                   # logits, gap, g
TOL_GATE_W = 1e-5                                   # absolute, weights in [0, 1]


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def make_inputs(shape, B, seed, rho=0.5, router_std=None, alphas=None, layer=0, wl_id=0,
                w_std=0.02, margin=True, experts=True):
    router = gen.make_router(shape, seed, layer, wl_id, router_std)
    rej = None
    if margin:
        r = oracle.margin_reject(shape.top_k, shape.cap, alphas or (shape.alpha,), shape.act,
                                 shape.flags)
        rej = lambda x, w: r(x, w, router)  # noqa: E731
    x, conf_w, _ = gen.make_batch(shape, B, seed, layer, wl_id, rho, rej)
    d = {"x": x, "conf_w": conf_w, "router": router}
    if experts:
        d["experts"] = gen.make_experts(shape, seed, layer, wl_id, w_std)
        d["shared"] = gen.make_shared_experts(shape, seed, layer, wl_id, w_std)
    return d


def run_gpu(shape, d, dev_weights=None, packed=False, fused=False):
    """One pass through the C ABI; returns (host results, device weights).
    With packed=True the weights are re-laid by s2moe_pack_weights first and
    the layer carries S2MOE_PACKED_WEIGHTS (dev_weights are then the packed
    ones).  fused=True: the pass is one s2moe_moe_layer call instead of the
    four calls (route, gate, verify, combine)."""
    import torch

    import paper_2608_15018_amd as s2

    B = d["x"].shape[0]
    L = s2.make_layer(shape, flags=shape.flags | (s2.PACKED_WEIGHTS if packed else 0))
    p = s2.VerifyPass(L, B, fused=fused)
    x = s2.to_device(d["x"])
    router = s2.to_device(d["router"])
    conf = s2.to_device(d["conf_w"])
    if dev_weights is None:
        dev_weights = s2.weights_to_device(d["experts"], d["shared"])
        if packed:
            dev_weights = s2.pack_expert_weights(dev_weights[0], shape.wdt)
    p(x, router, conf, dev_weights[1])
    torch.cuda.synchronize()
    return p.results(), dev_weights


def assert_same_bits(a: dict, b: dict, label: str = ""):
    """Every output of two passes equal bit for bit."""
    assert a.keys() == b.keys(), label
    for n in a:
        x, y = np.asarray(a[n]), np.asarray(b[n])
        if x.dtype.kind == "f":
            same = x.shape == y.shape and np.array_equal(x.view(np.uint32), y.view(np.uint32))
        else:
            same = np.array_equal(x, y)
        assert same, f"{label}: {n} differs"


def rel_err(got, ref) -> float:
    ref = np.asarray(ref, dtype=np.float64)
    scale = np.abs(ref).max()
    return float(np.abs(np.asarray(got, dtype=np.float64) - ref).max() / (scale if scale else 1.0))


def check_routing(got: dict, ref: dict, label: str = ""):
    np.testing.assert_array_equal(got["plain_idx"], ref["plain_idx"], err_msg=label + " plain_idx")
    np.testing.assert_array_equal(got["pref"], ref["pref"], err_msg=label + " pref")
    np.testing.assert_array_equal(got["idx"], ref["idx"], err_msg=label + " idx")
    np.testing.assert_array_equal(got["count"], ref["count"], err_msg=label + " count")
    np.testing.assert_array_equal(got["offset"], ref["offset"], err_msg=label + " offset")
    np.testing.assert_array_equal(got["slot"], ref["slot"], err_msg=label + " slot")
    np.testing.assert_array_equal(got["uniq"], ref["uniq"], err_msg=label + " uniq")
    assert got["n_uniq"] == ref["n_uniq"], label + " n_uniq"
    assert rel_err(got["logits"], ref["logits"]) <= TOL_ROUTER, label + " logits"
    assert rel_err(got["gap"], ref["gap"]) <= TOL_ROUTER, label + " gap"
    assert rel_err(got["g"], ref["g"]) <= TOL_ROUTER, label + " g"
    assert np.abs(got["gate_w"] - ref["gate_w"]).max() <= TOL_GATE_W, label + " gate_w"


def check_outputs(got: dict, ref: dict, wdt: str, label: str = "") -> dict:
    e_out = rel_err(got["expert_out"], ref["expert_out"])
    e_y = rel_err(got["y"], ref["y"])
    tol = TOL_Y[wdt]
    assert np.isfinite(got["y"]).all(), label + " non-finite y"
    assert e_out <= tol, f"{label} expert_out max-rel {e_out:.3e} > {tol}"
    assert e_y <= tol, f"{label} y max-rel {e_y:.3e} > {tol}"
    return {"expert_out": e_out, "y": e_y}
