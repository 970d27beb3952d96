"""Invariants of reuse-aware gating that follow from the paper's definitions
(Sec. "Reuse-aware Expert Gating"), checked on the oracle over random inputs,
plus the worked-example analog and the paper's printed tables."""

import os

import numpy as np
import pytest

import oracle
from oracle import s2moe_oracle as O
from synth.configs import WORKLOADS

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _case(seed, B=None, E=None, k=None, cap=None, rho=0.5):
    rng = np.random.default_rng(seed)
    E = E or int(rng.integers(4, 40))
    k = k or int(rng.integers(1, max(2, E // 3)))
    cap = cap or int(rng.integers(k, E + 1))
    B = B or int(rng.integers(1, 24))
    shared = rng.standard_normal(E)
    ell = np.sqrt(rho) * shared + np.sqrt(1 - rho) * rng.standard_normal((B, E))
    w = rng.random(B)
    r = {"logits": ell, "plain_idx": np.array([O.top_k_ascending(v, k) for v in ell]),
         "gap": np.array([np.sort(v)[::-1][0] - np.sort(v)[::-1][k] for v in ell])}
    return ell, w, r, k, cap


def _gate(ell, w, r, k, cap, alpha, flags=0):
    return oracle.reuse_gate(ell, r["gap"], r["plain_idx"], w, k, cap, alpha, flags)


SEEDS = range(40)


@pytest.mark.parametrize("seed", SEEDS)
def test_I1_zero_alpha_is_plain_topk(seed):
    ell, w, r, k, cap = _case(seed)
    np.testing.assert_array_equal(_gate(ell, w, r, k, cap, 0.0)["idx"], r["plain_idx"])


@pytest.mark.parametrize("seed", SEEDS)
def test_I2_cap_equal_E_is_plain_topk(seed):
    ell, w, r, k, _ = _case(seed)
    E = ell.shape[1]
    np.testing.assert_array_equal(_gate(ell, w, r, k, E, 0.7)["idx"], r["plain_idx"])


@pytest.mark.parametrize("seed", SEEDS)
def test_I3_single_token_is_plain_topk(seed):
    ell, w, r, k, cap = _case(seed, B=1)
    np.testing.assert_array_equal(_gate(ell, w, r, k, cap, 1.5)["idx"], r["plain_idx"])


@pytest.mark.parametrize("seed", SEEDS)
def test_I4_identical_tokens_give_k_unique_experts(seed):
    ell, w, r, k, cap = _case(seed)
    B = ell.shape[0]
    ell = np.tile(ell[:1], (B, 1))
    r = {"logits": ell, "plain_idx": np.tile(r["plain_idx"][:1], (B, 1)),
         "gap": np.full(B, r["gap"][0])}
    gt = _gate(ell, w, r, k, cap, 0.9)
    assert gt["n_uniq"] == k


@pytest.mark.parametrize("seed", SEEDS)
def test_I5_weights_sum_to_one_and_ids_distinct(seed):
    ell, w, r, k, cap = _case(seed)
    gt = _gate(ell, w, r, k, cap, 0.5)
    np.testing.assert_allclose(gt["gate_w"].sum(1), 1.0, rtol=0, atol=1e-14)
    assert all(len(set(row)) == k for row in gt["idx"])
    assert np.all(np.diff(gt["idx"], axis=1) > 0)          # ascending ids
    assert np.all(gt["gate_w"] > 0)


@pytest.mark.parametrize("seed", SEEDS)
def test_I6_selected_experts_in_plain_or_preferred(seed):
    ell, w, r, k, cap = _case(seed)
    gt = _gate(ell, w, r, k, cap, 1.3)
    pref = set(np.nonzero(gt["pref"])[0])
    for b in range(ell.shape[0]):
        assert set(gt["idx"][b]) <= set(r["plain_idx"][b]) | pref


@pytest.mark.parametrize("seed", SEEDS)
def test_I7_scale_and_shift_invariance(seed):
    ell, w, r, k, cap = _case(seed)
    base = _gate(ell, w, r, k, cap, 0.6)
    rng = np.random.default_rng(seed + 999)
    shift = rng.integers(-4, 5, size=ell.shape[0]).astype(np.float64)
    ell2 = ell + shift[:, None]
    r2 = dict(r, logits=ell2)
    g2 = _gate(ell2, 3.0 * w, r2, k, cap, 0.6)
    np.testing.assert_array_equal(g2["pref"], base["pref"])
    np.testing.assert_array_equal(g2["idx"], base["idx"])
    np.testing.assert_allclose(g2["gate_w"], base["gate_w"], rtol=1e-12)


@pytest.mark.parametrize("seed", SEEDS)
def test_I8_activated_only_never_adds_experts(seed):
    ell, w, r, k, cap = _case(seed)
    gt = _gate(ell, w, r, k, cap, 2.0, oracle.PREF_ACTIVATED_ONLY)
    plain_u = set(np.unique(r["plain_idx"]))
    assert set(np.unique(gt["idx"])) <= plain_u
    assert gt["n_uniq"] <= len(plain_u)
    assert gt["pref"].sum() <= cap


@pytest.mark.parametrize("seed", SEEDS)
def test_I9_top1_kept_for_alpha_at_most_one(seed):
    ell, w, r, k, cap = _case(seed)
    for alpha in (0.25, 0.5, 0.99):
        gt = _gate(ell, w, r, k, cap, alpha)
        for b in range(ell.shape[0]):
            assert int(np.argmax(ell[b])) in set(gt["idx"][b])


@pytest.mark.parametrize("seed", SEEDS)
def test_I10_token_permutation_equivariance(seed):
    ell, w, r, k, cap = _case(seed)
    base = _gate(ell, w, r, k, cap, 0.8)
    p = np.random.default_rng(seed).permutation(ell.shape[0])
    rp = {"logits": ell[p], "plain_idx": r["plain_idx"][p], "gap": r["gap"][p]}
    gp = _gate(ell[p], w[p], rp, k, cap, 0.8)
    np.testing.assert_array_equal(gp["pref"], base["pref"])
    np.testing.assert_array_equal(gp["idx"], base["idx"][p])
    np.testing.assert_allclose(gp["gate_w"], base["gate_w"][p], rtol=1e-12)
    assert gp["n_uniq"] == base["n_uniq"]


def test_nonpositive_confidences_disable_the_bias():
    ell, w, r, k, cap = _case(3)
    gt = _gate(ell, -np.abs(w), r, k, cap, 5.0)
    assert gt["pref"].sum() == 0
    np.testing.assert_array_equal(gt["idx"], r["plain_idx"])
    gz = _gate(ell, np.zeros_like(w), r, k, cap, 5.0)
    np.testing.assert_array_equal(gz["idx"], r["plain_idx"])


def test_worked_example_analog():
    """Analog of the paper's illustration of reuse-aware gating (Fig. "An
    illustrative example of reuse-aware expert gating with top-2 routing"):
    4 draft tokens of decreasing confidence, 8 experts, top-2, a preferred set
    of 3 experts; the bias cuts the activated experts from 6 to 4, the two
    most confident tokens keep their choices and the least confident one
    moves into the preferred set.  The figure's numbers are not in the text,
    so these logits are constructed to show the same behaviour."""
    ell = np.array([[3.0, 2.5, 1.0, 0.2, 0.1, 0.0, -0.5, -1.0],
                    [2.8, 0.4, 2.6, 0.3, 0.2, 0.1, -0.5, -1.0],
                    [1.0, 2.4, 0.5, 2.0, 0.1, 0.0, -0.5, -1.0],
                    [0.3, 0.2, 1.5, 0.0, 2.0, 1.7, -0.5, -1.0]])
    w = np.array([0.9, 0.8, 0.5, 0.2])
    r = oracle.route(ell.astype(np.float32), np.eye(8, dtype=np.float32), 2, "f32")
    gt = oracle.reuse_gate(r["logits"], r["gap"], r["plain_idx"], w, 2, 3, 0.8)
    assert set(np.nonzero(gt["pref"])[0]) == {0, 1, 2}
    assert len(np.unique(r["plain_idx"])) == 6
    assert gt["n_uniq"] == 4
    np.testing.assert_array_equal(gt["idx"][:2], r["plain_idx"][:2])
    assert set(gt["idx"][3]) - set(r["plain_idx"][3]) == {2}
    assert 2 in set(np.nonzero(gt["pref"])[0])


def _read_table(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def test_golden_reuse_improvement_is_relative_reduction():
    rows = _read_table("expert_reuse.txt")
    assert len(rows) == 2
    for _, without, with_rg, pct in rows:
        assert float(with_rg) < float(without)
        val = oracle.reuse_improvement(float(without), float(with_rg))
        assert round(val, 2) == float(pct)


def test_golden_model_table_caps_and_workloads():
    rows = {r[0]: tuple(int(v) for v in r[1:]) for r in _read_table("model_draft_configs.txt")}
    for E, k, cap, draft in rows.values():
        assert k <= cap <= E              # TopCap requires cap >= k
        assert 1 <= draft < k             # the draft activates fewer experts
    qwen, deepseek = rows["Qwen3"], rows["DeepSeek"]
    c3, c4 = WORKLOADS["c3"].shape, WORKLOADS["c4"].shape
    assert (c3.n_experts, c3.top_k, c3.cap) == qwen[:3]
    assert (c4.n_experts, c4.top_k, c4.cap) == deepseek[:3]
