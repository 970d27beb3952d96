"""GPU checks of s2moe_moe_layer, one MoE layer in one call.

* Bit for bit equal to s2moe_route, s2moe_reuse_gate, s2moe_verify_moe and
  s2moe_combine called in turn, in every routing array, expert_out and y:
  on batches that take the three-launch path (B <= 4 with alpha = 0, or one
  token; bf16 and int4 weights; E of 8 to 200, so one, two or four experts
  per lane in the ranking; shared experts; down K split over 1 and 4 waves;
  packed and row-major weights) and on batches that do not (alpha > 0 at
  B = 2, too many segments, B = 8, B = 16, fp32 weights).
* The number of launches, read from a captured HIP graph: 3 on the fused
  path against 6 (bf16) or 7 (int4: x to fp16 is a launch of its own) for
  the same layer as four calls; one fewer than the four calls where the
  gating launch ranks the logits itself; with int4 weights also without the
  x conversion and the K parts' reduce; the same count where the routing
  ranks in its own workgroups or the logits are too many to stage.
* Against the oracle on the fused cases (routing exact, outputs within the
  bf16 tolerance), and graph replays equal to the eager call.
"""

import ctypes

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


def _shape(**kw):
    base = dict(hidden=256, ffn=512, n_experts=8, top_k=2, cap=2, alpha=0.0, act="bf16",
                wdt="bf16")
    base.update(kw)
    return LayerShape(**base)


# (label, shape, B, takes the three-launch path)
CASES = [
    ("e8 k2 B1", _shape(), 1, True),
    ("e8 k2 B4", _shape(), 4, True),
    ("e64 k3 B3 shared", _shape(hidden=512, ffn=256, n_experts=64, top_k=3, cap=3, n_shared=2,
                                ffn_shared=256), 3, True),
    ("e128 k3 B1", _shape(hidden=512, n_experts=128, top_k=3, cap=3), 1, True),
    ("e200 k4 B2", _shape(ffn=384, n_experts=200, top_k=4, cap=4), 2, True),
    ("F2048 KW4 B1", _shape(ffn=2048, n_experts=16, top_k=3, cap=3), 1, True),
    ("alpha B1", _shape(n_experts=32, top_k=4, cap=8, alpha=0.7), 1, True),
    ("alpha flags B1", _shape(n_experts=32, top_k=4, cap=8, alpha=0.5, flags=1 | 4), 1, True),
    ("alpha B2 (four calls)", _shape(n_experts=32, top_k=4, cap=8, alpha=0.7), 2, False),
    ("k16 B4 (four calls)", _shape(n_experts=64, top_k=16, cap=16), 4, False),
    ("F2048 B2 (four calls)", _shape(ffn=2048, n_experts=16, top_k=3, cap=3), 2, False),
    ("B8 (four calls)", _shape(), 8, False),
    ("int4 B2", _shape(wdt="q4g32"), 2, True),
    ("fp32 B1 (four calls)", _shape(act="f32", wdt="f32"), 1, False),
    ("B16 E8 (route_kernel)", _shape(cap=4, alpha=0.5), 16, False),
    ("int4 e64 k3 B4 shared", _shape(hidden=512, ffn=256, n_experts=64, top_k=3, cap=3,
                                     n_shared=2, ffn_shared=256, wdt="q4g32"), 4, True),
    ("int4 e128 k3 B1 F1024", _shape(hidden=512, ffn=1024, n_experts=128, top_k=3, cap=3,
                                     wdt="q4g32"), 1, True),
    ("int4 alpha B1", _shape(n_experts=32, top_k=4, cap=8, alpha=0.7, wdt="q4g32"), 1, True),
    ("int4 alpha B2 (four calls)", _shape(n_experts=32, top_k=4, cap=8, alpha=0.7,
                                          wdt="q4g32"), 2, False),
    ("B64 E256 (unstaged gate)", _shape(ffn=256, n_experts=256, top_k=4, cap=8, alpha=0.5), 64,
     False),
    ("int4 B16 K parts", _shape(ffn=8192, cap=4, alpha=0.5, wdt="q4g32"), 16, False),
    ("int4 B12 E96 K parts rows", _shape(hidden=128, ffn=4096, n_experts=96, cap=4, alpha=0.5,
                                         wdt="q4g32"), 12, False),
]


def _poison(p):
    for t in list(vars(p.rt).values()) + [p.expert_out, p.y]:
        if isinstance(t, torch.Tensor):
            t.fill_(float("nan") if t.is_floating_point() else -7)


def _run(shape, d, fused, packed):
    import paper_2608_15018_amd as s2
    from paper_2608_15018_amd.pipeline import pack_expert_weights, to_device, weights_to_device
    B = d["x"].shape[0]
    layer = s2.make_layer(shape, flags=shape.flags | (s2.PACKED_WEIGHTS if packed else 0))
    dev, w = weights_to_device(d["experts"], d["shared"])
    if packed:
        dev, w = pack_expert_weights(dev, shape.wdt)
    p = s2.VerifyPass(layer, B, fused=fused)
    _poison(p)
    ins = (to_device(d["x"]), to_device(d["router"]), to_device(d["conf_w"]))
    torch.cuda.synchronize()
    p(*ins, w)
    torch.cuda.synchronize()
    return p, ins, w, dev


def _assert_same(a: dict, b: dict, label):
    for n in a:
        x, y = np.asarray(a[n]), np.asarray(b[n])
        if x.dtype.kind == "f":
            assert np.array_equal(x.view(np.uint32), y.view(np.uint32)), f"{label}: {n} differs"
        else:
            assert np.array_equal(x, y), f"{label}: {n} differs"


def _graph_kernel_nodes(fn) -> int:
    """Kernel launches of fn(), captured into a HIP graph and counted."""
    g = torch.cuda.CUDAGraph(keep_graph=True)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        fn()
    hip = ctypes.CDLL("libamdhip64.so")
    n = ctypes.c_size_t(0)
    assert hip.hipGraphGetNodes(ctypes.c_void_p(g.raw_cuda_graph()), None, ctypes.byref(n)) == 0
    return int(n.value)


# Every case with row-major weights, and again packed where the weights can be
# (the packed layout exists for bf16 and int4 weights only).
LAYOUTS = [(c, False) for c in CASES] + [(c, True) for c in CASES if c[1].wdt != "f32"]


@pytest.mark.parametrize("case,packed", LAYOUTS,
                         ids=[f"{c[0]}-{'packed' if p else 'rows'}" for c, p in LAYOUTS])
def test_moe_layer_equals_four_calls(case, packed):
    label, shape, B, fused = case
    d = make_inputs(shape, B, seed=31 + B + shape.n_experts, rho=0.5)
    tag = f"{label} packed={packed}"
    log(f"[moe_layer] {tag}: H={shape.hidden} F={shape.ffn} E={shape.n_experts} "
        f"k={shape.top_k} S={shape.n_shared} B={B} wdt={shape.wdt}")
    p1, ins, w, _dev1 = _run(shape, d, fused=True, packed=packed)
    p4, _, _, _dev4 = _run(shape, d, fused=False, packed=packed)
    got1, got4 = p1.results(), p4.results()
    _assert_same(got1, got4, tag)
    if fused:
        ex, sh, sref = d["experts"], d["shared"], shape
        if shape.wdt == "q4g32":
            deq = lambda e: {n: np.stack([oracle.dequant_q4g32(e[n][i], e[n + "_s"][i])  # noqa: E731
                                          for i in range(e[n].shape[0])]).astype(np.float32)
                             for n in ("gate", "up", "down")} if e else {}
            ex, sh, sref = deq(ex), deq(sh), shape.with_(wdt="f32")
        ref = oracle.forward(d["x"], d["router"], d["conf_w"], ex, sh, sref)
        check_routing(got1, ref, tag)
        check_outputs(got1, ref, shape.wdt, tag)
    log(f"[moe_layer] {tag}: equal, n_uniq={got1['n_uniq']}")


# (case, launches of one call, launches of the four calls).  Three on the
# fused path; elsewhere the gating launch ranks the logits itself where the
# routing would rank them in a launch of its own (B <= 8 or E > 64, logits
# staged in LDS or a single-wave gate, up to 16 tokens), and with int4
# weights the routing launch also converts x and the combine launch also
# adds the down projection's K parts.
LAUNCHES = [(1, 3, 6), (2, 3, 6), (8, 5, 6), (12, 3, 7), (14, 5, 5), (19, 6, 6), (15, 3, 7),
            (18, 5, 7), (20, 5, 7), (21, 5, 8)]


@pytest.mark.parametrize("case,n_call,n_four", LAUNCHES, ids=[CASES[c[0]][0] for c in LAUNCHES])
def test_moe_layer_launch_count(case, n_call, n_four):
    import paper_2608_15018_amd as s2
    label, shape, B, _fused = CASES[case]
    d = make_inputs(shape, B, seed=5, rho=0.5)
    p1, ins, w, _dev = _run(shape, d, fused=True, packed=True)
    n1 = _graph_kernel_nodes(lambda: p1(*ins, w))
    p4 = s2.VerifyPass(p1.layer, B, fused=False)
    n4 = _graph_kernel_nodes(lambda: p4(*ins, w))
    log(f"[moe_layer] {label}: {n1} launches in one call, {n4} as four calls")
    assert (n1, n4) == (n_call, n_four)


@pytest.mark.parametrize("case", [2, 20, 14], ids=[CASES[c][0] for c in (2, 20, 14)])
def test_moe_layer_graph_replays(case):
    """Replays of a captured call, with eager work and synchronisations in
    between, equal the eager call bit for bit: a fused call, an int4 call
    whose combine launch adds the K parts, and a 16-token bf16 call."""
    label, shape, B, _fused = CASES[case]
    d = make_inputs(shape, B, seed=77, rho=0.5)
    p, ins, w, _dev = _run(shape, d, fused=True, packed=True)
    eager = p.results()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        p(*ins, w)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        p(*ins, w)
    for rep in range(3):
        _poison(p)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        _assert_same(p.results(), eager, f"{label} replay {rep}")
        p(*ins, w)
        torch.cuda.synchronize()
    log(f"[moe_layer] {label}: graph replays equal the eager call")


def _random_case(rng):
    """A random layer and batch inside the ABI limits, small enough for the
    host generator: both sides of the three-launch boundary."""
    wdt = rng.choice(["bf16", "bf16", "q4g32", "f32"])
    mult = 128 if wdt == "q4g32" else 64
    E = int(rng.choice([4, 8, 16, 33, 64, 100, 128, 200]))
    k = int(rng.integers(1, min(E - 1, 16) + 1))
    cap = int(rng.integers(k, min(E, 3 * k) + 1))
    S = int(rng.choice([0, 0, 1, 2]))
    shape = LayerShape(hidden=mult * int(rng.integers(1, 5)), ffn=mult * int(rng.integers(1, 9)),
                       n_experts=E, top_k=k, cap=cap, alpha=float(rng.choice([0.0, 0.0, 0.6])),
                       n_shared=S, ffn_shared=mult * int(rng.integers(1, 5)) if S else 0,
                       flags=int(rng.choice([0, 0, 1, 4, 7])),
                       act="f32" if wdt == "f32" else "bf16", wdt=wdt)
    B = int(rng.choice([1, 1, 2, 3, 4, 4, 5, 8, 12]))
    return shape, B


@pytest.mark.parametrize("seed", range(24))
def test_moe_layer_random_shapes(seed):
    """Random layers (E 4-200, k 1-16, shared experts, fp32/bf16/int4,
    flags, alpha 0 or 0.6, B 1-12): one call equals the four calls bit for
    bit in every output."""
    rng = np.random.default_rng(1000 + seed)
    shape, B = _random_case(rng)
    d = make_inputs(shape, B, seed=seed, rho=0.5)
    packed = shape.wdt != "f32" and bool(seed % 2)
    tag = (f"random {seed}: H={shape.hidden} F={shape.ffn} E={shape.n_experts} k={shape.top_k} "
           f"cap={shape.cap} S={shape.n_shared} B={B} a={shape.alpha} flags={shape.flags} "
           f"{shape.wdt} packed={packed}")
    log(f"[moe_layer] {tag}")
    p1, _, _, _d1 = _run(shape, d, fused=True, packed=packed)
    p4, _, _, _d4 = _run(shape, d, fused=False, packed=packed)
    _assert_same(p1.results(), p4.results(), tag)
