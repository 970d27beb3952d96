"""GPU checks of the expert-sparse draft pass (paper_2608_15018_amd.draft).

* Parity against the oracle at k_draft = 1, 2, 3 with no reuse bias, for
  one to four draft tokens, bf16 and int4 weights, with and without shared
  experts: routing bit-exact, outputs within the bf16/int4 tolerance.
* The four model shapes of the paper's table (one layer, B = 1, weights
  drawn on the device): routing against the oracle and the outputs of the
  experts actually used.
* A multi-layer draft step captured in a HIP graph: every replay, with
  eager work and synchronisations in between, equals the eager step bit for
  bit.
"""

import numpy as np
import pytest

import oracle
from synth import gen
from synth.configs import LayerShape
from tests.gpu_helpers import check_outputs, check_routing, log

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_15018_amd as s2
    s2.load()


def _small(k_draft, wdt, shared):
    return LayerShape(hidden=256, ffn=512, n_experts=16, top_k=k_draft, cap=k_draft, alpha=0.0,
                      n_shared=2 if shared else 0, ffn_shared=256 if shared else 0,
                      act="bf16", wdt=wdt)


def _run_layer(shape, d, packed):
    import paper_2608_15018_amd as s2
    from paper_2608_15018_amd.pipeline import pack_expert_weights, to_device, weights_to_device
    B = d["x"].shape[0]
    layer = s2.make_layer(shape, flags=s2.PACKED_WEIGHTS if packed else 0)
    dev, w = weights_to_device(d["experts"], d["shared"])
    if packed:
        dev, w = pack_expert_weights(dev, shape.wdt)
    p = s2.VerifyPass(layer, B)
    p(to_device(d["x"]), to_device(d["router"]), to_device(d["conf_w"]), w)
    torch.cuda.synchronize()
    return p.results()


@pytest.mark.parametrize("wdt", ["bf16", "q4g32"])
@pytest.mark.parametrize("k_draft", [1, 2, 3])
@pytest.mark.parametrize("shared", [False, True])
def test_draft_layer_parity(wdt, k_draft, shared):
    shape = _small(k_draft, wdt, shared)
    for B in (1, 2, 4):
        seed = 100 * k_draft + B
        router = gen.make_router(shape, seed)
        rej = oracle.margin_reject(k_draft, k_draft, (0.0,), "bf16")
        x, conf, _ = gen.make_batch(shape, B, seed, rho=0.3,
                                    reject=lambda xx, ww: rej(xx, ww, router))
        d = {"x": x, "router": router, "conf_w": conf,
             "experts": gen.make_experts(shape, seed), "shared": gen.make_shared_experts(shape, seed)}
        label = f"draft k={k_draft} B={B} {wdt} shared={shared}"
        log(f"[draft] {label}")
        got = _run_layer(shape, d, packed=True)
        if wdt == "q4g32":
            deq = lambda ex: {n: np.stack([oracle.dequant_q4g32(ex[n][e], ex[n + "_s"][e])  # noqa: E731
                                           for e in range(ex[n].shape[0])]).astype(np.float32)
                              for n in ("gate", "up", "down")} if ex else {}
            ref = oracle.forward(x, router, conf, deq(d["experts"]), deq(d["shared"]),
                                 shape.with_(wdt="f32"))
        else:
            ref = oracle.forward(x, router, conf, d["experts"], d["shared"], shape)
        check_routing(got, ref, label)
        assert (got["idx"] == got["plain_idx"]).all(), "no bias: the draft routes plain top-k"
        check_outputs(got, ref, wdt, label)


@pytest.mark.parametrize("model", ["olmoe", "deepseek", "qwen3", "gptoss"])
def test_model_shaped_draft_layers(model):
    """One draft layer of each model shape at B = 1; the oracle sees the
    same bytes (host copies of the experts the token uses)."""
    import paper_2608_15018_amd as s2
    from paper_2608_15018_amd import draft
    from synth import device_gen
    m = draft.DRAFT_MODELS[model]
    k, E, H, F = m["k_draft"], m["n_experts"], m["hidden"], m["ffn"]
    S, Fs = m.get("n_shared", 0), m.get("ffn_shared", 0)
    layer = draft.draft_layer(model, packed=False)
    ex = device_gen.expert_weights(E, F, H, "bf16", seed=7, layer=0)
    sh = device_gen.expert_weights(S, Fs, H, "bf16", seed=7, layer=0, tag=1) if S else {}
    x = device_gen.activations(1, H, seed=7, layer=0, rho=0.0)
    router = device_gen.router(E, H, seed=7, layer=0)
    p = s2.VerifyPass(layer, 1)
    p(x, router, torch.ones(1, device="cuda"), s2.make_weights(ex, sh))
    torch.cuda.synchronize()
    got = p.results()
    bits = lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)  # noqa: E731
    xh, rh = bits(x), bits(router)
    shape = LayerShape(hidden=H, ffn=F, n_experts=E, top_k=k, cap=k, alpha=0.0, n_shared=S,
                       ffn_shared=Fs, act="bf16", wdt="bf16")
    r = oracle.route(xh, rh, k, "bf16")
    lg = np.sort(r["logits"][0])[::-1]
    assert lg[k - 1] - lg[k] > 1e-4, "routing too close to a tie for an exact check"
    np.testing.assert_array_equal(got["plain_idx"], r["plain_idx"])
    np.testing.assert_array_equal(got["idx"], r["plain_idx"])
    used = got["uniq"][: got["n_uniq"]]
    experts = {n: np.zeros((E,) + tuple(ex[n].shape[1:]), dtype=np.uint16) for n in ex}
    for n in ex:
        experts[n][used] = bits(ex[n][torch.as_tensor(used, device="cuda").long()])
    shared = {n: bits(v) for n, v in sh.items()}
    ref = oracle.forward(xh, rh, np.ones(1, np.float32), experts, shared, shape)
    log(f"[draft] {model}: experts {used.tolist()}")
    check_routing(got, ref, model)
    check_outputs(got, ref, "bf16", model)


@pytest.mark.parametrize("wdt", ["bf16", "q4g32"])
def test_draft_step_graph_replays_match_eager(wdt):
    import paper_2608_15018_amd as s2
    from paper_2608_15018_amd.draft import DraftStep
    from paper_2608_15018_amd.pipeline import pack_expert_weights, to_device, weights_to_device
    shape = _small(2, wdt, shared=True)
    layer = s2.make_layer(shape, flags=s2.PACKED_WEIGHTS)
    inputs, keep = [], []
    for l in range(3):
        router = gen.make_router(shape, 5, l)
        x, _, _ = gen.make_batch(shape, 2, 5, l, rho=0.3)
        dev, w = weights_to_device(gen.make_experts(shape, 5, l), gen.make_shared_experts(shape, 5, l))
        dev, w = pack_expert_weights(dev, wdt)
        keep.append(dev)
        inputs.append((to_device(x), to_device(router), w))
    step = DraftStep(layer, 2, inputs)
    step()
    torch.cuda.synchronize()
    eager = [y.clone() for y in step.outputs()]
    eager_idx = [p.rt.idx.clone() for p in step.passes]
    step.capture()
    for rep in range(3):
        for y in step.outputs():
            y.fill_(float("nan"))
        torch.cuda.synchronize()
        step.replay()
        torch.cuda.synchronize()
        for l, y in enumerate(step.outputs()):
            assert torch.equal(y, eager[l]), f"replay {rep} layer {l}"
            assert torch.equal(step.passes[l].rt.idx, eager_idx[l])
        step()  # eager work between replays
        torch.cuda.synchronize()
        log(f"[draft] graph replay {rep} ok ({wdt})")
