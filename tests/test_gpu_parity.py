"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Routing decisions (plain_idx, pref, idx, count, offset, slot, uniq,
n_uniq) must match bit for bit; the inputs are drawn so that every ranking
decision is separated by >= 1e-3 (in fp64, on the stored values), which makes
the decision the same in fp32 and fp64.  Floating-point outputs must be
within the stated tolerances (max-abs error over max-abs reference).
"""

import numpy as np
import pytest

import oracle
from synth.configs import WORKLOAD_ID, WORKLOADS, LayerShape
from tests.gpu_helpers import (TOL_GATE_W, assert_same_bits, check_outputs, check_routing, log,
                               make_inputs, rel_err, run_gpu)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_15018_amd as s2
    s2.load()


def _oracle(shape, d):
    return oracle.forward(d["x"], d["router"], d["conf_w"], d["experts"], d["shared"], shape)


def _full_check(shape, d, label):
    log(f"[parity] {label}: B={d['x'].shape[0]} H={shape.hidden} F={shape.ffn} "
        f"E={shape.n_experts} k={shape.top_k} S={shape.n_shared} wdt={shape.wdt}")
    got, dw = run_gpu(shape, d)
    ref = _oracle(shape, d)
    check_routing(got, ref, label)
    errs = check_outputs(got, ref, shape.wdt, label)
    # The one-call layer (s2moe_moe_layer) on the same inputs and weights.
    one, _ = run_gpu(shape, d, dw, fused=True)
    assert_same_bits(one, got, f"{label} one call")
    log(f"[parity] {label}: ok n_uniq={got['n_uniq']} errs={errs}, one call equal")
    return got, ref


# Reduced shapes that keep each workload's routing structure and still span
# several 64-row blocks, several K blocks and ragged token tiles.
SMALL = {
    "c1": (WORKLOADS["c1"].shape, 8, 0.0, 0.02),
    "c2s": (LayerShape(hidden=512, ffn=1024, n_experts=8, top_k=2, cap=4, alpha=0.5), 16, 0.6,
            None),
    "c3s": (LayerShape(hidden=256, ffn=256, n_experts=128, top_k=8, cap=14, alpha=0.5), 32,
            0.5, None),
    "c4s": (LayerShape(hidden=256, ffn=192, n_experts=64, top_k=6, n_shared=2, ffn_shared=128,
                       cap=16, alpha=0.5), 64, 0.4, None),
    "c5s": (LayerShape(hidden=512, ffn=768, n_experts=8, top_k=2, cap=4, alpha=0.5,
                       wdt="q4g32"), 16, 0.6, None),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_small_workloads(name):
    shape, B, rho, rstd = SMALL[name]
    d = make_inputs(shape, B, seed=101, rho=rho, router_std=rstd)
    _full_check(shape, d, name)


@pytest.mark.parametrize("alpha", [0.0, 0.5, 1.0])
def test_alpha_sweep_small(alpha):
    shape = SMALL["c3s"][0].with_(alpha=alpha)
    d = make_inputs(shape, 32, seed=7, rho=0.5, alphas=(alpha,))
    got, ref = _full_check(shape, d, f"c3s alpha={alpha}")
    if alpha == 0.0:
        np.testing.assert_array_equal(got["idx"], got["plain_idx"])


@pytest.mark.parametrize("B", [1, 4, 8, 12, 16, 64])
def test_int4_draft_sizes_small(B):
    shape = SMALL["c5s"][0]
    d = make_inputs(shape, B, seed=300 + B, rho=0.6)
    _full_check(shape, d, f"c5s B={B}")


@pytest.mark.parametrize("flags", [1, 2, 4, 7])
def test_gating_variants(flags):
    shape = SMALL["c3s"][0].with_(flags=flags, alpha=0.8)
    d = make_inputs(shape, 32, seed=50 + flags, rho=0.5, alphas=(0.8,))
    _full_check(shape, d, f"flags={flags}")


def test_single_token():
    shape = SMALL["c2s"][0]
    d = make_inputs(shape, 1, seed=3, rho=0.6)
    got, _ = _full_check(shape, d, "B=1")
    np.testing.assert_array_equal(got["idx"], got["plain_idx"])


@pytest.mark.parametrize("B,E,k,cap,H,F,S,wdt", [
    (13, 7, 3, 5, 320, 192, 0, "bf16"),
    (37, 25, 4, 9, 192, 320, 1, "bf16"),
    (5, 11, 2, 4, 384, 256, 0, "q4g32"),
    (23, 13, 3, 6, 256, 384, 1, "q4g32"),
])
def test_odd_expert_counts_and_batches(B, E, k, cap, H, F, S, wdt):
    """Expert counts that fill no 4- or 16-expert group, batch sizes that
    fill no token tile, and (with S = 1) a shared expert of another width:
    the routing kernels' partial expert groups and the FFN tails."""
    shape = LayerShape(hidden=H, ffn=F, n_experts=E, top_k=k, cap=cap, alpha=0.5,
                       n_shared=S, ffn_shared=F + 128 if S else 0, wdt=wdt)
    d = make_inputs(shape, B, seed=900 + B, rho=0.5)
    _full_check(shape, d, f"odd B={B} E={E} k={k} {wdt}")


@pytest.mark.parametrize("B,E,k,cap,act", [
    (24, 96, 4, 8, "f32"),
    (40, 130, 5, 10, "bf16"),
    (9, 200, 8, 20, "f32"),
])
def test_router_rows_path_many_experts(B, E, k, cap, act):
    """Batches over more than 64 experts take the two-launch router (one wave
    per router row and token, then one wave per token ranking) at any B:
    fp32 and bf16 activations, an expert count that fills no 4-expert group
    (130) and one that needs four experts per lane in the ranking (200)."""
    shape = LayerShape(hidden=256, ffn=128, n_experts=E, top_k=k, cap=cap, alpha=0.5,
                       act=act, wdt=act)
    d = make_inputs(shape, B, seed=1300 + B, rho=0.5)
    _full_check(shape, d, f"router rows B={B} E={E} {act}")


@pytest.mark.parametrize("B", [1, 2, 4])
@pytest.mark.parametrize("alpha", [0.0, 0.7])
@pytest.mark.parametrize("flags", [0, 1, 2, 4, 7])
@pytest.mark.parametrize("E,k,cap", [(8, 2, 4), (64, 6, 16), (200, 8, 20)])
def test_small_batch_gating(B, alpha, flags, E, k, cap):
    """Draft-sized batches (the single-wave gating path when alpha = 0 or
    B = 1): every routing output against the oracle, for each reading of
    the gating and expert counts in all three per-lane slot widths."""
    shape = LayerShape(hidden=256, ffn=128, n_experts=E, top_k=k, cap=cap, alpha=alpha,
                       flags=flags)
    d = make_inputs(shape, B, seed=1000 + 7 * B + E + flags, rho=0.5)
    got, ref = _full_check(shape, d, f"small B={B} alpha={alpha} flags={flags} E={E}")
    if alpha == 0.0 or B == 1:
        np.testing.assert_array_equal(got["idx"], got["plain_idx"])


def test_max_tokens_one_hot_expert_load():
    """B = 256 (the ABI maximum) with strongly shared routing, so single
    experts receive far more than 64 tokens (several token passes)."""
    shape = LayerShape(hidden=256, ffn=256, n_experts=8, top_k=2, cap=4, alpha=0.5)
    d = make_inputs(shape, 256, seed=9, rho=0.95)
    got, _ = _full_check(shape, d, "B=256")
    assert got["count"].max() > 64


def test_max_experts_and_topk():
    shape = LayerShape(hidden=128, ffn=128, n_experts=256, top_k=16, cap=40, alpha=0.5)
    d = make_inputs(shape, 24, seed=4, rho=0.5)
    _full_check(shape, d, "E=256 k=16")


def test_max_tokens_experts_and_topk_together():
    """B = 256 with E = 256 and k = 16: 4096 assignments, logits too many
    to stage in LDS, every bucket-building path at its largest."""
    shape = LayerShape(hidden=128, ffn=128, n_experts=256, top_k=16, cap=48, alpha=0.5)
    d = make_inputs(shape, 256, seed=12, rho=0.5)
    got, _ = _full_check(shape, d, "B=256 E=256 k=16")
    assert got["count"].sum() == 256 * 16


def test_int4_deepseek_shaped_with_shared():
    """int4 weights at the DeepSeek-V2-Lite expert width F = F_s = 1408
    (11 super-steps of 128, not a power of two) with 2 shared experts,
    packed and row-major, at 4 and 64 tokens."""
    shape = LayerShape(hidden=512, ffn=1408, n_experts=16, top_k=6, n_shared=2, ffn_shared=1408,
                       cap=12, alpha=0.5, act="bf16", wdt="q4g32")
    for B in (4, 64):
        d = make_inputs(shape, B, seed=21 + B, rho=0.4)
        deq = lambda ex: {n: np.stack([oracle.dequant_q4g32(ex[n][e], ex[n + "_s"][e])  # noqa: E731
                                       for e in range(ex[n].shape[0])]).astype(np.float32)
                          for n in ("gate", "up", "down")}
        log(f"[parity] int4 F=1408 shared B={B}")
        got, _ = run_gpu(shape, d)
        packed, _ = run_gpu(shape, d, packed=True)
        assert np.array_equal(packed["expert_out"], got["expert_out"])
        ref = oracle.forward(d["x"], d["router"], d["conf_w"], deq(d["experts"]),
                             deq(d["shared"]), shape.with_(wdt="f32"))
        check_routing(got, ref, f"int4 F=1408 B={B}")
        check_outputs(got, ref, "q4g32", f"int4 F=1408 B={B}")


@pytest.mark.parametrize("hidden,B,seed", [(384, 48, 71), (640, 40, 62), (512, 64, 63)])
def test_int4_row_split_gate_up(hidden, B, seed):
    """Above 16 tokens the int4 gate-up runs on the row-split kernel with
    LDS-staged activations: hidden sizes of 3, 5 and 4 super-steps (an odd
    count ends on a half chunk), buckets of up to 16, 17-32 and more than 32
    tokens (two passes over the rows), a shared expert in one case; packed
    equal to row-major bit for bit, outputs against the oracle."""
    S = 1 if hidden == 640 else 0
    shape = LayerShape(hidden=hidden, ffn=256, n_experts=8, top_k=2, cap=4, alpha=0.5,
                       n_shared=S, ffn_shared=128 if S else 0, act="bf16", wdt="q4g32")
    d = make_inputs(shape, B, seed=seed, rho=0.6)
    label = f"int4 row-split H={hidden} B={B}"
    log(f"[parity] {label}")
    got, _ = run_gpu(shape, d)
    packed, _ = run_gpu(shape, d, packed=True)
    counts = np.asarray(got["count"])
    assert counts.max() > 32 and ((counts > 16) & (counts <= 32)).any(), counts
    assert np.array_equal(packed["expert_out"], got["expert_out"]), label
    assert np.array_equal(packed["y"], got["y"]), label
    deq = lambda ex: {n: np.stack([oracle.dequant_q4g32(ex[n][e], ex[n + "_s"][e])  # noqa: E731
                                   for e in range(ex[n].shape[0])]).astype(np.float32)
                      for n in ("gate", "up", "down")} if ex else {}
    ref = oracle.forward(d["x"], d["router"], d["conf_w"], deq(d["experts"]), deq(d["shared"]),
                         shape.with_(wdt="f32"))
    check_routing(got, ref, label)
    check_outputs(got, ref, "q4g32", label)


def _bf16_scaled(bits, factor):
    """bf16 bit patterns times a power of two (exact away from the ends of
    the range, which the test's values stay clear of)."""
    f = (bits.astype(np.uint32) << 16).view(np.float32) * np.float32(factor)
    u = f.view(np.uint32)
    assert not (u & 0xFFFF).any()
    return (u >> 16).astype(np.uint16)


@pytest.mark.parametrize("B,seed", [(4, 81), (64, 82)])
def test_int4_fp16_range_large_magnitudes(B, seed):
    """int4 weights with values near the top of the fp16 range the header
    allows: x times 2^12 (|x| up to about 1.6e4) and the router times 2^-12,
    which leaves every logit, and so the routing, exactly as drawn; gate and
    up scales times 2^-5, so the SwiGLU activations Hh reach 1.2e4-1.8e4.
    B = 4 runs the K-split kernel, B = 64 the row-split one with four token
    tiles; packed equal to row-major bit for bit; outputs against the
    oracle at the int4 tolerance."""
    from oracle.s2moe_oracle import silu
    shape = LayerShape(hidden=256, ffn=512, n_experts=8, top_k=2, cap=4, alpha=0.5, act="bf16",
                       wdt="q4g32")
    d = make_inputs(shape, B, seed=seed, rho=0.5)
    d["x"] = _bf16_scaled(d["x"], 4096.0)
    d["router"] = _bf16_scaled(d["router"], 1.0 / 4096.0)
    ex = d["experts"]
    for n in ("gate_s", "up_s"):
        s16 = (ex[n].astype(np.float32) / 32).astype(np.float16)
        assert np.array_equal(s16.astype(np.float32) * 32, ex[n].astype(np.float32))
        ex[n] = s16
    W = {n: np.stack([oracle.dequant_q4g32(ex[n][e], ex[n + "_s"][e])
                      for e in range(shape.n_experts)]) for n in ("gate", "up", "down")}
    x = oracle.upcast(d["x"], "bf16")
    hh = silu(np.einsum("bh,efh->ebf", x, W["gate"])) * np.einsum("bh,efh->ebf", x, W["up"])
    x_max, hh_max = float(np.abs(x).max()), float(np.abs(hh).max())
    assert x_max >= 1.2e4 and 1e4 <= hh_max < 65504 / 2, (x_max, hh_max)
    label = f"int4 fp16 range B={B} |x|max={x_max:.0f} |Hh|max={hh_max:.0f}"
    log(f"[parity] {label}")
    got, _ = run_gpu(shape, d)
    packed, _ = run_gpu(shape, d, packed=True)
    assert np.array_equal(packed["expert_out"], got["expert_out"]), label
    ref = oracle.forward(d["x"], d["router"], d["conf_w"],
                         {n: w.astype(np.float32) for n, w in W.items()}, {},
                         shape.with_(wdt="f32"))
    check_routing(got, ref, label)
    errs = check_outputs(got, ref, "q4g32", label)
    log(f"[parity] {label}: ok errs={errs}")


def test_max_hidden():
    """H = 16384 (the documented maximum): long router rows and gate-up
    rows, bf16, small B."""
    shape = LayerShape(hidden=16384, ffn=256, n_experts=8, top_k=2, cap=4, alpha=0.5)
    for B in (3, 40):
        d = make_inputs(shape, B, seed=13 + B, rho=0.5)
        _full_check(shape, d, f"H=16384 B={B}")


@pytest.mark.parametrize("wdt", ["bf16", "q4g32"])
def test_max_ffn(wdt):
    """F = 262144 (the documented maximum): 4096 gate-up row blocks per
    expert and a down projection over 2048 super-steps of K; with int4
    weights the down launch splits K into its largest count of parts (8)."""
    shape = LayerShape(hidden=128, ffn=262144, n_experts=2, top_k=1, cap=1, alpha=0.5, wdt=wdt)
    d = make_inputs(shape, 12, seed=41, rho=0.5)
    _full_check(shape, d, f"F=262144 {wdt}")


@pytest.mark.parametrize("wdt", ["bf16", "q4g32"])
def test_max_shared_experts(wdt):
    """S = 8 shared experts (the ABI maximum) beside 16 routed ones, with
    F_s > F, so Hh rows are F_s wide and expert_out holds rows B k + s B + b
    for every s."""
    shape = LayerShape(hidden=256, ffn=256, n_experts=16, top_k=2, n_shared=8, ffn_shared=384,
                       cap=4, alpha=0.5, wdt=wdt)
    d = make_inputs(shape, 20, seed=31, rho=0.5)
    got, _ = _full_check(shape, d, f"S=8 {wdt}")
    assert got["expert_out"].shape[0] == 20 * 2 + 8 * 20


def test_cap_equal_E_and_identical_tokens():
    shape = LayerShape(hidden=256, ffn=256, n_experts=16, top_k=3, cap=16, alpha=0.9)
    d = make_inputs(shape, 12, seed=5, rho=0.5)
    got, _ = _full_check(shape, d, "cap=E")
    np.testing.assert_array_equal(got["idx"], got["plain_idx"])
    shape2 = shape.with_(cap=6)
    d2 = dict(d, x=np.tile(d["x"][:1], (12, 1)))
    got2, _ = _full_check(shape2, d2, "identical tokens")
    assert got2["n_uniq"] == 3


@pytest.mark.parametrize("kind", ["zero", "negative", "mixed"])
def test_degenerate_confidences(kind):
    shape = SMALL["c3s"][0]
    d = make_inputs(shape, 32, seed=21, rho=0.5)
    w = d["conf_w"].copy()
    if kind == "zero":
        w[:] = 0
    elif kind == "negative":
        w = -w
    else:
        w[::2] = -w[::2]
    d["conf_w"] = w.astype(np.float32)
    if kind == "mixed":
        # redraw so the margins hold for the changed confidences
        r = oracle.margin_reject(shape.top_k, shape.cap, (shape.alpha,), shape.act)
        from synth import gen
        d["x"], _, _ = gen.make_batch(shape, 32, 21, 0, 0, 0.5,
                                      lambda x, _w: r(x, d["conf_w"], d["router"]))
    got, _ = _full_check(shape, d, f"conf {kind}")
    if kind != "mixed":
        assert got["pref"].sum() == 0
        np.testing.assert_array_equal(got["idx"], got["plain_idx"])


def test_deterministic_bitwise():
    shape = SMALL["c4s"][0]
    d = make_inputs(shape, 64, seed=77, rho=0.4)
    a, dw = run_gpu(shape, d)
    b, _ = run_gpu(shape, d, dw)
    for n in ("logits", "gap", "g", "gate_w", "expert_out", "y"):
        assert np.array_equal(a[n], b[n]), n
    for n in ("idx", "slot", "uniq"):
        np.testing.assert_array_equal(a[n], b[n])


def test_exact_ties_resolved_by_lower_index():
    """Dyadic logits (exact in fp32 and fp64) with many exact ties, written
    straight into the logits buffer; only reuse_gate runs."""
    import paper_2608_15018_amd as s2
    rng = np.random.default_rng(0)
    B, E, k, cap = 32, 24, 4, 8
    ell = rng.integers(-8, 8, size=(B, E)).astype(np.float64) / 4.0   # many ties
    w = rng.integers(0, 5, size=B).astype(np.float32) / 4.0
    plain = np.array([oracle.s2moe_oracle.top_k_ascending(r, k) for r in ell], np.int32)
    gap = np.array([np.sort(r)[::-1][0] - np.sort(r)[::-1][k] for r in ell])
    for alpha, flags in ((0.5, 0), (1.0, 0), (0.25, 2), (0.5, 1)):
        ref = oracle.reuse_gate(ell, gap, plain, w, k, cap, alpha, flags)
        L = s2.make_layer(hidden=64, ffn=64, n_experts=E, top_k=k, cap=cap, alpha=alpha,
                          flags=flags)
        rt = s2.Routing(L, B)
        rt.logits.copy_(torch.from_numpy(ell.astype(np.float32)))
        rt.gap.copy_(torch.from_numpy(gap.astype(np.float32)))
        rt.plain_idx.copy_(torch.from_numpy(plain))
        s2.reuse_gate(L, torch.from_numpy(w).cuda(), rt)
        torch.cuda.synchronize()
        got = rt.host()
        for n in ("pref", "idx", "count", "offset", "slot", "uniq"):
            np.testing.assert_array_equal(got[n], ref[n], err_msg=f"{n} alpha={alpha} f={flags}")
        np.testing.assert_array_equal(got["g"], ref["g"].astype(np.float32))
        assert np.abs(got["gate_w"] - ref["gate_w"]).max() <= 1e-6


@pytest.mark.parametrize("B,E,k,cap", [(16, 8, 2, 4), (32, 128, 8, 14), (64, 64, 6, 16),
                                       (200, 256, 16, 40)])
def test_near_ties_sharing_upper_key_bits(B, E, k, cap):
    """Logits +-(1 + c 2^-16) with c < 96 all share the upper 16 bits of
    their order keys, so every top-k boundary falls inside one radix bucket
    and is settled by the exact in-bucket ranking; codes repeat, so exact
    ties occur too.  Weights are 0/1 and alpha is dyadic, so g, the bias
    and the biased logits are exact in fp32 and fp64.  Route runs on x with
    a one-hot fp32 router (logits = x exactly), then reuse_gate."""
    import paper_2608_15018_amd as s2
    rng = np.random.default_rng(B * 1000 + E)
    codes = rng.integers(0, 96, size=(B, E))
    sign = np.where(rng.random((B, E)) < 0.3, -1.0, 1.0)
    ell = sign * (1.0 + codes * 2.0 ** -16)
    H = max(64, -(-E // 64) * 64)
    x = np.zeros((B, H), np.float32)
    x[:, :E] = ell
    router = np.zeros((E, H), np.float32)
    router[np.arange(E), np.arange(E)] = 1.0
    w = (rng.random(B) < 0.6).astype(np.float32)
    w[0] = 1.0
    r_ref = oracle.route(x, router, k, "f32")
    for alpha, flags in ((0.5, 0), (1.0, 4), (0.5, 1)):
        ref = oracle.reuse_gate(r_ref["logits"], r_ref["gap"], r_ref["plain_idx"], w, k, cap,
                                alpha, flags)
        L = s2.make_layer(hidden=H, ffn=64, n_experts=E, top_k=k, cap=cap, alpha=alpha,
                          flags=flags, act="f32", wdt="f32")
        rt = s2.Routing(L, B)
        s2.route(L, torch.from_numpy(x).cuda(), torch.from_numpy(router).cuda(), rt)
        s2.reuse_gate(L, torch.from_numpy(w).cuda(), rt)
        torch.cuda.synchronize()
        got = rt.host()
        label = f"B={B} E={E} alpha={alpha} flags={flags}"
        np.testing.assert_array_equal(got["logits"], ell.astype(np.float32), err_msg=label)
        np.testing.assert_array_equal(got["plain_idx"], r_ref["plain_idx"], err_msg=label)
        np.testing.assert_array_equal(got["gap"], r_ref["gap"].astype(np.float32), err_msg=label)
        for n in ("pref", "idx", "count", "offset", "slot", "uniq"):
            np.testing.assert_array_equal(got[n], ref[n], err_msg=f"{n} {label}")
        np.testing.assert_array_equal(got["g"], ref["g"].astype(np.float32), err_msg=label)
        assert np.abs(got["gate_w"] - ref["gate_w"]).max() <= TOL_GATE_W, label


@pytest.mark.parametrize("nbytes", [16, 4096 + 48, (64 << 20) + 16 * 7])
def test_stream_read_touches_every_byte_once(nbytes):
    """The diagnostic read stream covers the buffer exactly once: the XOR of
    its per-block checksum words equals the XOR of all 32-bit words."""
    import paper_2608_15018_amd as s2
    rng = np.random.default_rng(nbytes)
    host = rng.integers(0, 1 << 32, size=nbytes // 4, dtype=np.uint32)
    buf = torch.from_numpy(host.view(np.int32)).cuda()
    sink = torch.zeros(s2.STREAM_SINK_WORDS, dtype=torch.int32, device="cuda")
    s2.stream_read(buf, sink)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(host)


# ---------------------------------------------------------------- packed weights
def _expected_pack_bf16(m):
    """Reference tile order written out independently: tile (rt, s) of 16 rows
    x 32 columns, lane L -> row 16 rt + L % 16, columns 32 s + 8 (L // 16)."""
    n, rows, K = m.shape
    out = np.empty(m.size, dtype=m.dtype)
    pos = 0
    for i in range(n):
        for rt in range(rows // 16):
            for s in range(K // 32):
                for L in range(64):
                    r, c = 16 * rt + L % 16, 32 * s + 8 * (L // 16)
                    out[pos:pos + 8] = m[i, r, c:c + 8]
                    pos += 8
    return out.reshape(m.shape)


def _expected_pack_q4(codes, scales):
    n, rows, half = codes.shape
    K = 2 * half
    oc = np.empty(codes.size, dtype=codes.dtype)
    osc = np.empty(scales.size, dtype=scales.dtype)
    pc = ps = 0
    for i in range(n):
        for rt in range(rows // 16):
            for S in range(K // 128):
                for L in range(64):
                    r, g = 16 * rt + L % 16, 4 * S + L // 16
                    oc[pc:pc + 16] = codes[i, r, 16 * g:16 * g + 16]
                    osc[ps] = scales[i, r, g]
                    pc += 16
                    ps += 1
    return oc.reshape(codes.shape), osc.reshape(scales.shape)


def test_pack_layout():
    import paper_2608_15018_amd as s2
    rng = np.random.default_rng(1)
    m = rng.integers(0, 1 << 16, size=(2, 32, 96), dtype=np.uint16)
    got, _ = s2.pack_weights("bf16", s2.to_device(m))
    torch.cuda.synchronize()
    got = got.view(torch.int16).cpu().numpy().view(np.uint16)
    np.testing.assert_array_equal(got, _expected_pack_bf16(m))
    codes = rng.integers(0, 256, size=(2, 32, 128), dtype=np.uint8)
    scales = rng.standard_normal((2, 32, 8)).astype(np.float16)
    gc, gs = s2.pack_weights("q4g32", s2.to_device(codes), s2.to_device(scales))
    torch.cuda.synchronize()
    ec, es = _expected_pack_q4(codes, scales)
    np.testing.assert_array_equal(gc.cpu().numpy(), ec)
    np.testing.assert_array_equal(gs.cpu().numpy(), es)


@pytest.mark.parametrize("name", ["c2s", "c3s", "c4s", "c5s"])
def test_packed_weights_match_plain_bitwise(name):
    """The packed layout changes only where weights are read from: the MFMA
    sequence, hence every output bit, is the same as with plain weights."""
    shape, B, rho, rstd = SMALL[name]
    d = make_inputs(shape, B, seed=404, rho=rho, router_std=rstd)
    plain, _ = run_gpu(shape, d)
    packed, _ = run_gpu(shape, d, packed=True)
    for n in ("idx", "slot", "uniq"):
        np.testing.assert_array_equal(packed[n], plain[n])
    assert np.array_equal(packed["expert_out"], plain["expert_out"]), name
    assert np.array_equal(packed["y"], plain["y"]), name
    check_outputs(packed, _oracle(shape, d), shape.wdt, name + " packed")


# ---------------------------------------------------------------- full sizes
def _workload_inputs(name, B, seed, layer=0, alphas=None):
    wl = WORKLOADS[name]
    return make_inputs(wl.shape, B, seed, rho=wl.rho, router_std=wl.router_std,
                       alphas=alphas or (wl.shape.alpha,), layer=layer,
                       wl_id=WORKLOAD_ID[name], w_std=wl.w_std)


def test_full_c2_mixtral_bf16():
    wl = WORKLOADS["c2"]
    d = _workload_inputs("c2", 16, seed=1)
    got, ref = _full_check(wl.shape, d, "c2 full")
    log(f"[parity] c2 reuse ratio {ref['reuse_ratio']:.3f}")
    packed, _ = run_gpu(wl.shape, d, packed=True)
    check_routing(packed, ref, "c2 full packed")
    errs = check_outputs(packed, ref, "bf16", "c2 full packed")
    log(f"[parity] c2 full packed ok errs={errs}")


def test_full_c3_alpha_sweep():
    wl = WORKLOADS["c3"]
    d = _workload_inputs("c3", 32, seed=1, alphas=wl.alphas)
    from paper_2608_15018_amd.pipeline import weights_to_device
    dw = weights_to_device(d["experts"], d["shared"])
    ratios = {}
    for alpha in wl.alphas:
        shape = wl.shape.with_(alpha=alpha)
        log(f"[parity] c3 full alpha={alpha}")
        got, _ = run_gpu(shape, d, dw)
        ref = _oracle(shape, d)
        check_routing(got, ref, f"c3 alpha={alpha}")
        check_outputs(got, ref, "bf16", f"c3 alpha={alpha}")
        one, _ = run_gpu(shape, d, dw, fused=True)
        assert_same_bits(one, got, f"c3 alpha={alpha} one call")
        ratios[alpha] = ref["reuse_ratio"]
    log(f"[parity] c3 reuse ratio by alpha: {ratios}")
    assert ratios[1.0] <= ratios[0.0]


def test_full_c4_shared_routed():
    wl = WORKLOADS["c4"]
    d = _workload_inputs("c4", 64, seed=1)
    _full_check(wl.shape, d, "c4 full")


@pytest.mark.parametrize("layer", [0, 11, 23])
def test_full_c5_int4_layers(layer):
    """Mixtral-shaped int4 layers 0, 11 and 23 of the 24-layer stack, each at
    draft sizes 1, 4, 16, 32 and 64 (every kernel configuration: the K-split
    kernel, then one, two and four token tiles per weight pass with 4, 4 and
    3 K parts of the down projection).  The oracle uses the exact fp32 values
    of the dequantised weights (s * (q - 8) has at most 15 significant bits)."""
    wl = WORKLOADS["c5"]
    sh = wl.shape
    dw = deq = None
    for B in (1, 4, 16, 32, 64):
        d = _workload_inputs("c5", B, seed=1, layer=layer)
        if dw is None:
            from paper_2608_15018_amd.pipeline import weights_to_device
            ex = d["experts"]
            deq = {n: np.stack([oracle.dequant_q4g32(ex[n][e], ex[n + "_s"][e]).astype(np.float32)
                                for e in range(sh.n_experts)])
                   for n in ("gate", "up", "down")}
            dw = weights_to_device(ex, {})
        log(f"[parity] c5 layer={layer} B={B}")
        got, _ = run_gpu(sh, d, dw)
        one, _ = run_gpu(sh, d, dw, fused=True)
        assert_same_bits(one, got, f"c5 l={layer} B={B} one call")
        if B in (16, 64):
            packed, _ = run_gpu(sh, d, packed=True)
            assert np.array_equal(packed["expert_out"], got["expert_out"])
        ref = oracle.forward(d["x"], d["router"], d["conf_w"], deq, {}, sh.with_(wdt="f32"))
        check_routing(got, ref, f"c5 l={layer} B={B}")
        errs = check_outputs(got, ref, "q4g32", f"c5 l={layer} B={B}")
        log(f"[parity] c5 layer={layer} B={B} ok n_uniq={got['n_uniq']} errs={errs}")
