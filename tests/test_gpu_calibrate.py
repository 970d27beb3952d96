"""The cost-model measurement (Sec. "Routing-aware Adaptive Speculative
Expansion": per activated expert cost T_exp, checked with R^2 and MAPE) on
the GPU: a tiny sweep of a small fine-grained layer (128 experts, top-8,
cap 14) at two batch sizes and two bias strengths.  Each sample's activated
expert count must equal the oracle's on the same inputs (drawn clear of
ranking ties), the latencies must be positive, and the fit must run."""

import numpy as np
import pytest

import oracle
from synth.configs import WORKLOADS, LayerShape
from tests.gpu_helpers import log

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_15018_amd as s2
    s2.load()


SHAPE = LayerShape(hidden=256, ffn=256, n_experts=128, top_k=8, cap=14, alpha=0.5)
BATCHES, ALPHAS, SEEDS = (8, 32), (0.0, 1.0), (3,)


def _reject_for(router, shape):
    r = oracle.margin_reject(shape.top_k, shape.cap, (shape.alpha,), shape.act, shape.flags)
    return lambda x, w: r(x, w, router)


def test_calibration_sweep_matches_oracle_expert_counts():
    from paper_2608_15018_amd import calibrate
    from synth import gen
    from synth.configs import WORKLOAD_ID

    log("[calibrate] tiny c3-shaped sweep")
    samples = calibrate.measure("c3", BATCHES, ALPHAS, SEEDS, steps=3, shape=SHAPE,
                                reject_for=_reject_for, rotate_bytes=0)
    assert len(samples) == len(BATCHES) * len(ALPHAS) * len(SEEDS)
    wl = WORKLOADS["c3"]
    for s in samples:
        shape = SHAPE.with_(alpha=s["alpha"])
        router, x, conf_w = calibrate.sample_inputs(
            wl, shape, s["B"], s["seed"], lambda r: _reject_for(r, shape))
        r = oracle.route(x, router, shape.top_k, shape.act)
        g = oracle.reuse_gate(r["logits"], r["gap"], r["plain_idx"], conf_w, shape.top_k,
                              shape.cap, shape.alpha, shape.flags)
        assert s["n_uniq"] == g["n_uniq"], s
        assert s["t_step_us"] > 0 and s["t_ffn_us"] > 0 and s["weight_copies"] == 1
        log(f"[calibrate] B={s['B']} alpha={s['alpha']} n_uniq={s['n_uniq']} ok")
    fit = calibrate.calibrate(samples)
    for k in ("step", "ffn"):
        assert np.isfinite(fit[k]["T_exp_us"]) and fit[k]["n"] == len(samples)
