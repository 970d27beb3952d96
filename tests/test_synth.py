"""The seeded input generators: determinism, stored formats, distributions."""

import numpy as np
import pytest
import torch

import oracle
from synth import gen
from synth.configs import WORKLOADS, LayerShape


def test_bf16_rounding_nearest_even_known_values():
    one_plus = np.float32(1.0) + np.float32(2.0 ** -8)          # halfway 1.0 / 1.0078125
    three_half = np.float32(1.0) + np.float32(3 * 2.0 ** -8)    # halfway 0x3F81 / 0x3F82
    a = np.array([1.0, -2.0, one_plus, three_half, -three_half, 3.14159265], np.float32)
    bits = gen.bf16_bits_from_f32(a)
    assert list(bits[:5]) == [0x3F80, 0xC000, 0x3F80, 0x3F82, 0xBF82]
    assert bits[5] == 0x4049


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    a = (rng.standard_normal(100_000) * np.exp(rng.uniform(-20, 20, 100_000))).astype(np.float32)
    ours = gen.bf16_bits_from_f32(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)


def test_same_seed_same_bytes_and_subset_consistency():
    sh = LayerShape(hidden=128, ffn=64, n_experts=6, top_k=2, cap=4)
    a = gen.make_experts(sh, 5)
    b = gen.make_experts(sh, 5)
    c = gen.make_experts(sh, 6)
    for n in ("gate", "up", "down"):
        np.testing.assert_array_equal(a[n], b[n])
        assert not np.array_equal(a[n], c[n])
    sub = gen.make_experts(sh, 5, experts=[4, 1])
    for n in ("gate", "up", "down"):
        np.testing.assert_array_equal(sub[n][0], a[n][4])
        np.testing.assert_array_equal(sub[n][1], a[n][1])
    x1, w1, _ = gen.make_batch(sh, 9, 3, rho=0.5)
    x2, w2, _ = gen.make_batch(sh, 9, 3, rho=0.5)
    np.testing.assert_array_equal(x1, x2)
    np.testing.assert_array_equal(w1, w2)


def test_q4_formats_and_value_distribution():
    sh = LayerShape(hidden=256, ffn=128, n_experts=2, top_k=1, cap=1, wdt="q4g32")
    ex = gen.make_experts(sh, 1)
    assert ex["gate"].dtype == np.uint8 and ex["gate"].shape == (2, 128, 128)
    assert ex["down"].shape == (2, 256, 64)
    assert ex["gate_s"].dtype == np.float16 and ex["gate_s"].shape == (2, 128, 8)
    w = oracle.dequant_q4g32(ex["gate"][0], ex["gate_s"][0])
    assert 0.015 < w.std() < 0.025
    lo = ex["gate"] & 0xF
    hi = ex["gate"] >> 4
    assert lo.min() == 0 and lo.max() == 15 and hi.min() == 0 and hi.max() == 15


def test_confidences_are_prefix_products():
    rng = np.random.default_rng(1)
    for B in (1, 4, 16, 20, 64):
        w = gen.draft_tree_confidence(B, rng)
        assert w.shape == (B,)
        assert np.all(w > 0) and np.all(w <= 1)
        D = min(8, B)
        for c in range(0, B, D):
            chain = w[c:c + D]
            assert np.all(np.diff(chain) <= 0)


def test_router_logit_correlation_close_to_rho():
    wl = WORKLOADS["c3"]
    sh = wl.shape
    router = gen.make_router(sh, 0, 0, 1, None)
    x, _, _ = gen.make_batch(sh, 32, 0, 0, 1, wl.rho)
    ell = oracle.upcast(x, "bf16") @ oracle.upcast(router, "bf16").T
    assert 0.8 < ell.std() < 1.2
    c = np.corrcoef(ell)
    off = c[~np.eye(32, dtype=bool)]
    assert abs(off.mean() - wl.rho) < 0.1


@pytest.mark.parametrize("name", ["c1", "c3", "c4"])
def test_margin_enforcement(name):
    wl = WORKLOADS[name]
    sh = wl.shape
    alphas = wl.alphas or (sh.alpha,)
    rej = oracle.margin_reject(sh.top_k, sh.cap, alphas, sh.act)
    d = gen.workload_inputs(wl, wl.batches[0], seed=11, reject=rej, with_experts=False)
    ell = oracle.upcast(d["x"], sh.act) @ oracle.upcast(d["router"], sh.act).T
    m = oracle.routing_margins(ell, d["conf_w"], sh.top_k, sh.cap, alphas)
    assert m["plain"].min() >= 1e-3
    assert m["cap_margin"] >= 1e-3
    for bm in m["biased"]:
        assert bm.min() >= 1e-3


# ------------------------------------------------------------- draft trees
def test_draft_trees_are_well_formed_and_seeded():
    from synth.trees import TREE_WORKLOADS, make_trees
    for wl in TREE_WORKLOADS.values():
        d = make_trees(wl, 3, seed=5)
        d2 = make_trees(wl, 3, seed=5)
        for k in d:
            np.testing.assert_array_equal(d[k], d2[k])
        N = wl.max_nodes
        assert d["parent"].shape == (3, N) and d["eid"].shape == (3, N, wl.n_layers, wl.k)
        for t in range(3):
            n = int(d["n_nodes"][t])
            assert wl.branch + (wl.depth - 1) * wl.beam_min * wl.branch <= n <= N
            par = d["parent"][t, :n]
            assert (par < np.arange(n)).all() and (par >= -1).all()
            q = d["q"][t, :n]
            assert ((q >= 0) & (q <= 1)).all()
            e = d["eid"][t, :n]
            assert ((e >= 0) & (e < wl.n_experts)).all()
            # k distinct experts per token and layer
            s = np.sort(e, axis=-1)
            assert (np.diff(s, axis=-1) > 0).all()
            assert (d["eid"][t, n:] == -1).all()
