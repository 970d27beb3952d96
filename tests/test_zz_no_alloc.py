"""s2moe_verify_moe_noalloc (the library's own scratch array) against
s2moe_verify_moe (a caller workspace) through the C ABI.

Each case makes two calls in a row on one layer, the second with fewer
tokens, so that the second call runs on scratch memory the first one left
behind.  Both entry points run the same kernels on the same inputs, so their
expert outputs must be equal bit for bit; the combined output is also checked
against the fp64 oracle at the usual tolerance."""

import numpy as np
import pytest

import oracle
from synth.configs import LayerShape
from tests.gpu_helpers import check_outputs, check_routing, log, make_inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_15018_amd as s2
    s2.load()


CASES = {
    "f32": (LayerShape(hidden=256, ffn=512, n_experts=8, top_k=2, cap=4, alpha=0.5,
                       act="f32", wdt="f32"), (8, 3), 0.0, 0.02, False),
    "bf16_shared": (LayerShape(hidden=256, ffn=192, n_experts=64, top_k=6, n_shared=2,
                               ffn_shared=128, cap=16, alpha=0.5), (64, 16), 0.4, None, False),
    "bf16_packed": (LayerShape(hidden=512, ffn=1024, n_experts=8, top_k=2, cap=4, alpha=0.5),
                    (32, 5), 0.6, None, True),
    "int4": (LayerShape(hidden=512, ffn=768, n_experts=8, top_k=2, cap=4, alpha=0.5,
                        wdt="q4g32"), (64, 4), 0.6, None, False),
    "int4_packed": (LayerShape(hidden=512, ffn=768, n_experts=8, top_k=2, cap=4, alpha=0.5,
                               wdt="q4g32"), (16, 1), 0.6, None, True),
    # Down projection in K parts, 3 at 16 tokens and 4 at 12 (partial sums in
    # the scratch array; 12 and 16 down items per expert).
    "int4_kparts": (LayerShape(hidden=512, ffn=4096, n_experts=8, top_k=2, cap=4, alpha=0.5,
                               wdt="q4g32"), (16, 12), 0.6, None, True),
    # Workspace of exactly the scratch size (512 rows of 16384 bf16), then 8 tokens.
    "at_limit": (LayerShape(hidden=256, ffn=16384, n_experts=8, top_k=2, cap=4, alpha=0.5),
                 (256, 8), 0.6, None, False),
}


def _call_pair(s2, shape, d, packed, dev_weights):
    B = d["x"].shape[0]
    L = s2.make_layer(shape, flags=shape.flags | (s2.PACKED_WEIGHTS if packed else 0))
    p = s2.VerifyPass(L, B)
    x = s2.to_device(d["x"])
    p.route(x, s2.to_device(d["router"]))
    p.reuse_gate(s2.to_device(d["conf_w"]))
    rows = B * shape.top_k + shape.n_shared * B
    eo_ws = torch.full((rows, shape.hidden), float("nan"), device="cuda")
    eo_na = torch.full((rows, shape.hidden), float("nan"), device="cuda")
    s2.verify_moe(L, x, dev_weights[1], p.rt, p.workspace, eo_ws)
    s2.verify_moe_noalloc(L, x, dev_weights[1], p.rt, eo_na)
    p.expert_out.copy_(eo_na)
    p.combine()
    torch.cuda.synchronize()
    got = p.results()
    return got, eo_ws.cpu().numpy(), eo_na.cpu().numpy()


@pytest.mark.parametrize("name", list(CASES))
def test_noalloc_matches_workspace_entry_point(name):
    import paper_2608_15018_amd as s2

    shape, batches, rho, rstd, packed = CASES[name]
    d0 = make_inputs(shape, batches[0], seed=4100, rho=rho, router_std=rstd)
    dev = s2.weights_to_device(d0["experts"], d0["shared"])
    if packed:
        dev = s2.pack_expert_weights(dev[0], shape.wdt)
    assert s2.workspace_bytes(s2.make_layer(shape), batches[0]) <= s2.NOALLOC_SCRATCH_BYTES
    for call, B in enumerate(batches):
        d = make_inputs(shape, B, seed=4100 + call, rho=rho, router_std=rstd, experts=False)
        d["experts"], d["shared"] = d0["experts"], d0["shared"]
        log(f"[noalloc] {name} call {call}: B={B} H={shape.hidden} F={shape.ffn} "
            f"E={shape.n_experts} wdt={shape.wdt} packed={packed}")
        got, eo_ws, eo_na = _call_pair(s2, shape, d, packed, dev)
        assert np.isfinite(eo_na).all(), f"{name} call {call}: unwritten expert_out rows"
        assert np.array_equal(eo_na, eo_ws), f"{name} call {call}: differs from s2moe_verify_moe"
        ref = oracle.forward(d["x"], d["router"], d["conf_w"], d["experts"], d["shared"], shape)
        check_routing(got, ref, f"{name} call {call}")
        errs = check_outputs(got, ref, shape.wdt, f"{name} call {call}")
        log(f"[noalloc] {name} call {call}: ok n_uniq={got['n_uniq']} errs={errs}")
