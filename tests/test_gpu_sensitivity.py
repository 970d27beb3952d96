"""GPU parity of the cap x alpha reuse sweep: every selection the sweep takes
from the library's routing and gating kernels equals the oracle's, on
margin-enforced batches of both layer shapes and every (cap, alpha) of the
grid."""

import numpy as np
import pytest

import oracle
from paper_2608_15018_amd import sensitivity as S
from synth import gen
from tests.gpu_helpers import log

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_15018_amd as s2
    s2.load()


@pytest.mark.parametrize("name", sorted(S.SHAPES))
@pytest.mark.parametrize("B", [8, 16])
def test_sweep_selections_match_oracle(name, B):
    s = S.SHAPES[name]
    k = s["top_k"]
    caps = S.caps_for(k, s["paper_cap"], s["n_experts"])
    for seed in (0, 1):
        shape = S.layer_shape(name, caps[0], 0.5)
        router = gen.make_router(shape, seed, 0, S.WL_ID)
        checks = [oracle.margin_reject(k, c, S.ALPHAS, "bf16") for c in caps]

        def reject(x, w):
            bad = np.zeros(x.shape[0], dtype=bool)
            for chk in checks:
                bad |= chk(x, w, router)
            return bad

        x, conf, rounds = gen.make_batch(shape, B, seed, 0, S.WL_ID, 0.2, reject)
        log(f"[sensitivity] {name} B={B} seed={seed} margin rounds={rounds}")
        got = S.gpu_selections(name, x, router, conf, caps, S.ALPHAS)
        r = oracle.route(x, router, k, "bf16")
        assert np.array_equal(got["plain_idx"], r["plain_idx"])
        for cap in caps:
            for alpha in S.ALPHAS:
                g = oracle.reuse_gate(r["logits"], r["gap"], r["plain_idx"], conf, k, cap, alpha)
                assert np.array_equal(got["idx"][(cap, alpha)], g["idx"]), (cap, alpha)
