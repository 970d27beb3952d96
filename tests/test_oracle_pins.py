"""Pins of the fp64 oracle against things other than itself.

Each test checks the oracle against brute force on tiny inputs, a closed
form, a textbook or library routine, or an invariant that follows from the
paper's definitions (Sec. "Reuse-aware Expert Gating").  They are chosen so
that a dropped term, a wrong sign or index, or a transposed operand in the
oracle fails at least one of them.
"""

import itertools
import math

import numpy as np
import pytest
from scipy.special import expit, softmax

import oracle
from oracle import s2moe_oracle as O


def _distinct(rng, shape, scale=1.0):
    """Random values whose sums over small subsets are pairwise distinct."""
    v = rng.standard_normal(shape) * scale
    return v + rng.random(shape) * 1e-3


def brute_topk(values, k):
    """Best k-subset by total value (unique when values are generic)."""
    best = max(itertools.combinations(range(len(values)), k),
               key=lambda s: sum(values[i] for i in s))
    return sorted(best)


# ---------------------------------------------------------------- route (a1, a2)
def check_router_orientation(O_mod):
    """W_r with unit rows e_{p(e)} gives ell_{b,e} = x_{b,p(e)}: pins the
    orientation ell = W_r x (a transposed router changes which coordinate is
    read)."""
    rng = np.random.default_rng(0)
    B, H, E = 5, 16, 6
    x = rng.standard_normal((B, H)).astype(np.float32)
    perm = np.array([3, 11, 0, 7, 15, 2])
    W = np.zeros((E, H), np.float32)
    W[np.arange(E), perm] = 1.0
    r = O_mod.route(x, W, 2, "f32")
    np.testing.assert_array_equal(r["logits"], x[:, perm].astype(np.float64))


def test_router_one_hot_rows_pick_coordinates():
    check_router_orientation(O)


def check_router_bf16(O_mod):
    """Logits on bf16 inputs equal the dot products of the decoded values;
    decoded values are checked against known bf16 encodings."""
    known = {0x3F80: 1.0, 0xC000: -2.0, 0x3F81: 1.0078125, 0x0000: 0.0,
             0x4049: 3.140625, 0xBF00: -0.5}
    for bits, val in known.items():
        assert O_mod.upcast(np.array([bits], np.uint16), "bf16")[0] == val
    x = np.array([[0x3F80, 0xC000, 0x4049]], np.uint16)     # [1, -2, 3.140625]
    W = np.array([[0x3F80, 0x3F80, 0x0000],                 # [1, 1, 0]
                  [0x0000, 0xBF00, 0x3F80]], np.uint16)     # [0, -0.5, 1]
    r = O_mod.route(x, W, 1, "bf16")
    np.testing.assert_array_equal(r["logits"], [[-1.0, 1.0 + 3.140625]])


def test_router_matches_explicit_loop_on_bf16_bits():
    check_router_bf16(O)


def check_plain_topk_and_gap(O_mod, seed):
    rng = np.random.default_rng(seed)
    E = int(rng.integers(3, 9))
    k = int(rng.integers(1, min(4, E)))
    B = int(rng.integers(1, 6))
    H = 8
    x = rng.standard_normal((B, H))
    W = rng.standard_normal((E, H))
    r = O_mod.route(x.astype(np.float32), W.astype(np.float32), k, "f32")
    for b in range(B):
        ell = list(r["logits"][b])
        assert list(r["plain_idx"][b]) == brute_topk(ell, k)
        desc = sorted(ell, reverse=True)
        assert r["gap"][b] == desc[0] - desc[k]          # top-1 minus (k+1)-th


@pytest.mark.parametrize("seed", range(20))
def test_plain_topk_and_gap_bruteforce(seed):
    check_plain_topk_and_gap(O, seed)


def check_ties(O_mod):
    ell = np.array([[1.0, 2.0, 2.0, 0.5, 2.0]])
    r_idx = O_mod.top_k_ascending(ell[0], 2)
    assert list(r_idx) == [1, 2]
    assert list(O_mod.rank_order(np.array([0.0, -0.0, 0.0]))) == [0, 1, 2]


def test_ties_break_toward_lower_expert_index():
    check_ties(O)


# ---------------------------------------------------------------- gating (a3-a5)
ACT_ONLY, ABSOLUTE, FROM_BIASED = 1, 2, 4      # the flag values of the C ABI


def brute_gate(ell, w, k, cap, alpha, flags=0):
    """Independent gating by subset enumeration, in plain Python floats.

    Sec. "Reuse-aware Expert Gating": confidences enter g only as
    non-negative weights, so w_b < 0 counts as 0 and, when no w_b is
    positive, no expert is preferred and no bias applies.  E* is the cap-subset
    of the candidates with the largest total g (the candidates are all experts,
    or with ACT_ONLY the union of the plain top-k sets; every candidate when
    there are at most cap of them).  The bias is alpha * (top-1 minus (k+1)-th
    logit), or alpha itself with ABSOLUTE.  The gate weights are exp(z_j) /
    sum_j exp(z_j) over the selected experts, z the original logits or, with
    FROM_BIASED, the biased ones."""
    B, E = ell.shape
    wc = [float(w[b]) if w[b] > 0 else 0.0 for b in range(B)]
    active = any(v > 0.0 for v in wc)
    g = [sum(wc[b] * float(ell[b][e]) for b in range(B)) for e in range(E)]
    plain = [brute_topk([float(v) for v in ell[b]], k) for b in range(B)]
    if not active:
        pref = set()
    else:
        cand = sorted(set().union(*map(set, plain))) if flags & ACT_ONLY else list(range(E))
        if len(cand) <= cap:
            pref = set(cand)
        else:
            pref = set(max(itertools.combinations(cand, cap),
                           key=lambda s: sum(g[e] for e in s)))
    idx, gw = [], []
    for b in range(B):
        row = [float(v) for v in ell[b]]
        desc = sorted(row, reverse=True)
        if not active:
            lam = 0.0
        elif flags & ABSOLUTE:
            lam = alpha
        else:
            lam = alpha * (desc[0] - desc[k])
        val = [row[e] + (lam if e in pref else 0.0) for e in range(E)]
        sel = brute_topk(val, k)
        src = val if flags & FROM_BIASED else row
        ez = [math.exp(src[e]) for e in sel]
        idx.append(sel)
        gw.append([v / sum(ez) for v in ez])
    return {"g": g, "pref": pref, "idx": idx, "gate_w": gw}


GATE_FLAGS = (0, ACT_ONLY, ABSOLUTE, FROM_BIASED, ACT_ONLY | ABSOLUTE | FROM_BIASED)
W_MODES = ("nonneg", "mixed", "nonpos")


def gate_case(seed, w_mode):
    """A small gating problem: logits with distinct subset sums, confidences
    drawn >= 0, of mixed sign (mostly one positive or more), or all <= 0."""
    rng = np.random.default_rng(100 + seed)
    E = int(rng.integers(4, 9))
    k = int(rng.integers(1, min(3, E - 1) + 1))
    cap = int(rng.integers(k, min(6, E) + 1))
    B = int(rng.integers(1, 7))
    alpha = float(rng.choice([0.0, 0.3, 0.5, 0.9, 2.0]))
    ell = _distinct(rng, (B, E))
    if w_mode == "nonneg":
        w = rng.random(B)
    elif w_mode == "mixed":
        w = rng.standard_normal(B)
        w[int(rng.integers(0, B))] = rng.random() + 0.1    # at least one positive
    else:
        w = -rng.random(B) * (rng.random(B) < 0.7)          # negatives and zeros
    return ell, w, k, cap, alpha


def check_gate_case(O_mod, seed, flags, w_mode):
    """Compare O_mod.reuse_gate with brute_gate on one case; raise
    AssertionError on any difference."""
    ell, w, k, cap, alpha = gate_case(seed, w_mode)
    desc = [sorted(row, reverse=True) for row in ell]
    gap = np.array([d[0] - d[k] for d in desc])
    plain = np.array([brute_topk(list(row), k) for row in ell])
    gt = O_mod.reuse_gate(ell, gap, plain, w, k, cap, alpha, flags)
    ref = brute_gate(ell, w, k, cap, alpha, flags)
    np.testing.assert_allclose(gt["g"], ref["g"], rtol=1e-12, atol=1e-12)
    assert set(np.nonzero(gt["pref"])[0]) == ref["pref"]
    assert [list(r) for r in gt["idx"]] == ref["idx"]
    np.testing.assert_allclose(gt["gate_w"], ref["gate_w"], rtol=1e-12, atol=0)
    # g pinned by one-hot confidences: g = 0.7 ell_b0, whatever the others'
    # (non-positive) values
    rng = np.random.default_rng(seed)
    b0 = int(rng.integers(0, ell.shape[0]))
    onehot = np.minimum(w, 0.0)
    onehot[b0] = 0.7
    g1 = O_mod.reuse_gate(ell, gap, plain, onehot, k, cap, alpha, flags)["g"]
    np.testing.assert_allclose(g1, 0.7 * ell[b0], rtol=0, atol=1e-15)


@pytest.mark.parametrize("w_mode", W_MODES)
@pytest.mark.parametrize("flags", GATE_FLAGS)
@pytest.mark.parametrize("seed", range(30))
def test_reuse_gate_bruteforce(seed, flags, w_mode):
    check_gate_case(O, seed, flags, w_mode)


def test_bias_is_alpha_times_top1_minus_kplus1_gap():
    """One token, E=5, k=2, E* forced to {3}.  Expert 3 enters the top-2 iff
    ell_3 + alpha*gap > ell_(2).  With ell = [3, 2, 1.5, 1, 0]: gap = 3 - 1.5,
    so expert 3 replaces expert 1 exactly when alpha > (2 - 1) / 1.5."""
    ell = np.array([[3.0, 2.0, 1.5, 1.0, 0.0],
                    [0.0, 0.0, 0.0, 50.0, 0.0]])   # token 1 pushes g_3 to the top
    w = np.array([0.0, 1.0])
    k, cap = 2, 2
    gap = np.array([1.5, 50.0])
    plain = np.array([[0, 1], [2, 3]])
    a_star = 1.0 / 1.5
    lo = oracle.reuse_gate(ell, gap, plain, w, k, cap, a_star - 1e-9)
    hi = oracle.reuse_gate(ell, gap, plain, w, k, cap, a_star + 1e-9)
    assert lo["pref"][3] == 1
    assert list(lo["idx"][0]) == [0, 1]
    assert list(hi["idx"][0]) == [0, 3]
    np.testing.assert_allclose(hi["lam"][0], (a_star + 1e-9) * 1.5)
    # absolute bias reading: lambda = alpha
    ab = oracle.reuse_gate(ell, gap, plain, w, k, cap, 1.0 + 1e-9, oracle.BIAS_ABSOLUTE)
    assert list(ab["idx"][0]) == [0, 3]
    ab = oracle.reuse_gate(ell, gap, plain, w, k, cap, 1.0 - 1e-9, oracle.BIAS_ABSOLUTE)
    assert list(ab["idx"][0]) == [0, 1]


def test_gate_weights_are_softmax_of_original_logits():
    rng = np.random.default_rng(7)
    B, E, k, cap = 6, 8, 3, 5
    ell = _distinct(rng, (B, E), 2.0)
    w = rng.random(B)
    gap = np.array([np.sort(r)[::-1][0] - np.sort(r)[::-1][k] for r in ell])
    plain = np.array([O.top_k_ascending(r, k) for r in ell])
    gt = oracle.reuse_gate(ell, gap, plain, w, k, cap, 0.8)
    for b in range(B):
        np.testing.assert_allclose(gt["gate_w"][b], softmax(ell[b, gt["idx"][b]]),
                                   rtol=1e-14, atol=0)
    gb = oracle.reuse_gate(ell, gap, plain, w, k, cap, 0.8, oracle.GATE_FROM_BIASED)
    for b in range(B):
        np.testing.assert_allclose(gb["gate_w"][b], softmax(gb["biased"][b, gb["idx"][b]]),
                                   rtol=1e-14, atol=0)


def check_bucketing(O_mod):
    rng = np.random.default_rng(3)
    for _ in range(20):
        E = int(rng.integers(2, 20))
        k = int(rng.integers(1, min(E, 5)))
        B = int(rng.integers(1, 40))
        idx = np.array([np.sort(rng.choice(E, k, replace=False)) for _ in range(B)])
        bk = O_mod.bucket(idx, E)
        flat = idx.reshape(-1)
        np.testing.assert_array_equal(bk["slot"], np.argsort(flat, kind="stable"))
        np.testing.assert_array_equal(bk["count"], np.bincount(flat, minlength=E))
        np.testing.assert_array_equal(bk["offset"][1:], np.cumsum(np.bincount(flat, minlength=E)))
        u = np.unique(flat)
        assert bk["n_uniq"] == u.size
        np.testing.assert_array_equal(bk["uniq"][:u.size], u)
        assert np.all(bk["uniq"][u.size:] == -1)
        assert bk["reuse_ratio"] == u.size / (B * k)


def test_bucketing_matches_stable_argsort():
    check_bucketing(O)


def check_route_and_bucket_pins(O_mod):
    """Every pin of the router, the plain top-k with its gap, the tie rule
    and the bucketing, run on one oracle module."""
    check_router_orientation(O_mod)
    check_router_bf16(O_mod)
    for seed in range(20):
        check_plain_topk_and_gap(O_mod, seed)
    check_ties(O_mod)
    check_bucketing(O_mod)


# ---------------------------------------------------------------- FFN (a7-a11)
def check_swiglu_identity(O_mod):
    """W_g = c I, W_u = I, W_d = P (a permutation): y = P (silu(c x) * x).
    Swapping gate and up gives silu(x) * c x, a transposed W_d gives P^T."""
    rng = np.random.default_rng(11)
    H = 8
    c = 1.75                       # exact in fp32
    x = rng.standard_normal((3, H)).astype(np.float32)
    P = np.eye(H)[[2, 5, 0, 7, 1, 3, 6, 4]]
    experts = {"gate": (c * np.eye(H))[None].astype(np.float32),
               "up": np.eye(H)[None].astype(np.float32),
               "down": P[None].astype(np.float32)}
    gt = {"idx": np.zeros((3, 1), np.int32)}
    out = O_mod.verify_moe(x, experts, {}, gt, 1, "f32", "f32")
    xd = x.astype(np.float64)
    expect = (c * xd * expit(c * xd) * xd) @ P.T
    np.testing.assert_allclose(out, expect, rtol=1e-14, atol=1e-15)


def test_swiglu_closed_form_identity_weights():
    check_swiglu_identity(O)


def check_down_linear(O_mod):
    rng = np.random.default_rng(12)
    H, F, E = 8, 16, 3
    x = rng.standard_normal((4, H)).astype(np.float32)
    ex = {n: rng.standard_normal((E, F, H)).astype(np.float32) for n in ("gate", "up")}
    ex["down"] = rng.standard_normal((E, H, F)).astype(np.float32)
    gt = {"idx": np.array([[0, 2], [1, 2], [0, 1], [2, 0]], np.int32)}
    base = O_mod.verify_moe(x, ex, {}, gt, 2, "f32", "f32")
    ex2 = dict(ex, down=ex["down"] * np.float32(2.0))
    np.testing.assert_allclose(O_mod.verify_moe(x, ex2, {}, gt, 2, "f32", "f32"), 2 * base,
                               rtol=1e-14)
    ex0 = dict(ex, down=np.zeros_like(ex["down"]))
    assert not O_mod.verify_moe(x, ex0, {}, gt, 2, "f32", "f32").any()


def test_down_projection_is_linear_and_zero_gives_zero():
    check_down_linear(O)


def check_dense_then_mask(O_mod, seed):
    """All experts on all tokens, then a one-hot gate mask (einsum-based)
    equals the oracle's grouped verify_moe + combine."""
    rng = np.random.default_rng(200 + seed)
    H, F, E, k, S, Fs = 16, 24, 6, 2, int(seed % 3), 8
    B = int(rng.integers(1, 9))
    x = rng.standard_normal((B, H)).astype(np.float32)
    ex = {"gate": rng.standard_normal((E, F, H)).astype(np.float32) * 0.3,
          "up": rng.standard_normal((E, F, H)).astype(np.float32) * 0.3,
          "down": rng.standard_normal((E, H, F)).astype(np.float32) * 0.3}
    sh = {"gate": rng.standard_normal((S, Fs, H)).astype(np.float32) * 0.3,
          "up": rng.standard_normal((S, Fs, H)).astype(np.float32) * 0.3,
          "down": rng.standard_normal((S, H, Fs)).astype(np.float32) * 0.3} if S else {}
    idx = np.array([np.sort(rng.choice(E, k, replace=False)) for _ in range(B)], np.int32)
    gw = rng.random((B, k))
    gw /= gw.sum(1, keepdims=True)
    eo = O_mod.verify_moe(x, ex, sh, {"idx": idx}, k, "f32", "f32", S)
    y = O_mod.combine(gw, eo, k, S)

    X = x.astype(np.float64)
    a = np.einsum("bh,efh->bef", X, ex["gate"].astype(np.float64))
    u = np.einsum("bh,efh->bef", X, ex["up"].astype(np.float64))
    dense = np.einsum("bef,ehf->beh", a * expit(a) * u, ex["down"].astype(np.float64))
    G = np.zeros((B, E))
    for b in range(B):
        G[b, idx[b]] = gw[b]
    ref = np.einsum("be,beh->bh", G, dense)
    for s in range(S):
        a = X @ sh["gate"][s].astype(np.float64).T
        ref += (a * expit(a) * (X @ sh["up"][s].astype(np.float64).T)) @ sh["down"][s].astype(np.float64).T
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(8))
def test_dense_then_mask_bruteforce(seed):
    check_dense_then_mask(O, seed)


def check_int4_known_codes(O_mod):
    """Byte 0x8F holds element 0 = 15 (low nibble) and element 1 = 8 (high);
    with scale 0.5: w = 0.5 * (15 - 8) = 3.5 and 0.5 * (8 - 8) = 0."""
    codes = np.zeros((2, 32), np.uint8)          # rows=2, K=64 -> 2 groups per row
    codes[0, 0] = 0x8F
    codes[0, 16] = 0x10                          # group 1: elem 32 = 0, elem 33 = 1
    codes[1, :] = 0x88                           # all exactly zero
    scales = np.array([[0.5, 0.25], [3.0, 7.0]], np.float16)
    w = O_mod.dequant_q4g32(codes, scales)
    assert w.shape == (2, 64)
    assert w[0, 0] == 3.5 and w[0, 1] == 0.0
    assert w[0, 2] == 0.5 * (0 - 8)
    assert w[0, 32] == 0.25 * (0 - 8) and w[0, 33] == 0.25 * (1 - 8)
    assert not w[1].any()


def test_int4_dequant_known_codes():
    check_int4_known_codes(O)


# ---------------------------------------------------------------- combine (a10)
def check_combine_small(O_mod):
    eo = np.array([[1.0, 2.0],     # token 0, slot 0
                   [10.0, 20.0],   # token 0, slot 1
                   [3.0, 4.0],     # token 1, slot 0
                   [30.0, 40.0],   # token 1, slot 1
                   [100.0, 0.0],   # shared 0, token 0
                   [0.0, 100.0]])  # shared 0, token 1
    gw = np.array([[0.25, 0.75], [0.5, 0.5]])
    y = O_mod.combine(gw, eo, 2, 1)
    np.testing.assert_array_equal(y, [[0.25 + 7.5 + 100.0, 0.5 + 15.0],
                                      [1.5 + 15.0, 2.0 + 20.0 + 100.0]])


def test_combine_small_numbers():
    check_combine_small(O)


def check_ffn_pins(O_mod):
    """Every pin of the expert FFN, dequantisation and combine steps, run on
    one oracle module (the oracle itself, or a copy with a planted mistake)."""
    check_swiglu_identity(O_mod)
    check_down_linear(O_mod)
    for seed in range(8):
        check_dense_then_mask(O_mod, seed)
    check_int4_known_codes(O_mod)
    check_combine_small(O_mod)


# ---------------------------------------------------------------- reuse ratio
def test_reuse_ratio_bounds_and_identical_tokens():
    """1/B <= r <= 1 (Sec. Motivation, Challenge 2: the ideal ratio is 1/s);
    identical tokens activate exactly k experts."""
    rng = np.random.default_rng(5)
    E, k = 16, 4
    for B in (1, 3, 8):
        idx = np.array([np.sort(rng.choice(E, k, replace=False)) for _ in range(B)])
        r = oracle.bucket(idx, E)["reuse_ratio"]
        assert 1.0 / B - 1e-15 <= r <= 1.0
        same = np.tile(idx[:1], (B, 1))
        bk = oracle.bucket(same, E)
        assert bk["n_uniq"] == k and bk["reuse_ratio"] == 1.0 / B
