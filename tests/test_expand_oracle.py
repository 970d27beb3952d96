"""Pins of the expansion oracle (Sec. "Routing-aware Adaptive Speculative
Expansion") against things other than itself: hand-derived trees, the
confidence-threshold rule it reduces to when new experts cost nothing, closed
forms on chains, exact scaling laws of U_i = B_i / C_i, and invariants of the
greedy selection checked with independent set arithmetic (numpy).

A dropped T_exp or C^draft term, a reversed set difference, a wrong prefix
product, a frontier that ignores the tree, a strict instead of a non-strict
threshold or a tie broken the other way fails at least one of them.
"""

import numpy as np
import pytest

from oracle import expand_oracle as X
from synth.trees import TREE_WORKLOADS, make_trees
from tests.expand_fixtures import load

DYADIC = np.array([1.0, 0.875, 0.75, 0.625, 0.5, 0.375, 0.25, 0.125], dtype=np.float32)


def run(tree_arrays, E, t_ar, t_exp, max_admit=0):
    parent, q, eid, c, root, n = tree_arrays
    return X.expand(parent, q, eid, c, E, t_ar, t_exp, root, n, max_admit)


@pytest.mark.parametrize("tree", load(), ids=lambda t: t.name)
def test_worked_examples(tree):
    r = run(tree.arrays(), tree.E, tree.t_ar, tree.t_exp, tree.max_admit)
    m = int(r["n_admit"][0])
    assert list(r["order"][0, :m]) == tree.expect["order"]
    assert list(r["util"][0, :m]) == tree.expect["util"]  # exact: dyadic inputs
    assert list(r["n_new"][0, :m]) == tree.expect["n_new"]
    assert int(r["n_pairs"][0]) == tree.expect["n_pairs"]
    assert int(r["status"][0]) == tree.expect["status"]
    # padding after the selected nodes
    assert (r["order"][0, m:] == -1).all() and (r["util"][0, m:] == 0).all()


def test_worked_examples_padded_layout_is_inert():
    """Padding slots beyond n_nodes are never looked at."""
    for tree in load():
        a = tree.arrays(n_pad=len(tree.nodes) + 5)
        a[0][0, len(tree.nodes):] = 99  # garbage parents in the padding
        r = run(a, tree.E, tree.t_ar, tree.t_exp, tree.max_admit)
        m = int(r["n_admit"][0])
        assert list(r["order"][0, :m]) == tree.expect["order"]
        assert int(r["status"][0]) == tree.expect["status"]


# ------------------------------------------------------------- random trees
def random_tree(rng, n, L, E, k, dyadic=False, root=True):
    parent = np.empty(n, dtype=np.int32)
    for i in range(n):
        parent[i] = rng.integers(-1, i) if i else -1
    if dyadic:
        q = DYADIC[rng.integers(0, len(DYADIC), n)]
    else:
        q = rng.random(n).astype(np.float32)
    eid = rng.integers(-1, E + 1, size=(n, L, k)).astype(np.int32)  # incl. padding ids
    c = (rng.random(n) * 4 + 0.5).astype(np.float32)
    r = rng.integers(0, E, size=(L, k)).astype(np.int32) if root else None
    return parent, q, eid, c, r


def batch1(parent, q, eid, c, r):
    n = len(parent)
    return (parent[None], q[None], eid[None], c[None], None if r is None else r[None],
            np.array([n], dtype=np.int32))


def pair_ids(eid_rows, E):
    """Independent set encoding: sorted unique l*E + e over valid ids."""
    L = eid_rows.shape[0]
    lay = np.repeat(np.arange(L), eid_rows.shape[1]).reshape(eid_rows.shape)
    ok = (eid_rows >= 0) & (eid_rows < E)
    return np.unique(lay[ok] * E + eid_rows[ok])


def path_product(parent, q, i):
    """p_i by walking up from i (leaf-up order; exact for dyadic q)."""
    p = 1.0
    while i >= 0:
        p *= float(q[i])
        i = int(parent[i])
    return p


def test_zero_expert_cost_is_confidence_threshold():
    """T_exp = 0 and one C^draft: U_i = p_i T_AR / c, so the greedy takes
    nodes by falling prefix confidence (ties: lower index) and keeps exactly
    those with p_i >= c / T_AR -- confidence-threshold pruning."""
    rng = np.random.default_rng(1)
    for trial in range(40):
        n = int(rng.integers(1, 40))
        parent, q, eid, c, r = random_tree(rng, n, 3, 8, 2, dyadic=True)
        c[:] = 1.0
        t_ar = float(2 ** rng.integers(1, 8))
        res = run(batch1(parent, q, eid, c, r), 8, t_ar, 0.0)
        p = np.array([path_product(parent, q, i) for i in range(n)])
        keep = [i for i in range(n) if p[i] * t_ar >= 1.0]
        want = sorted(keep, key=lambda i: (-p[i], i))
        m = int(res["n_admit"][0])
        assert list(res["order"][0, :m]) == want, trial
        np.testing.assert_array_equal(res["util"][0, :m], p[want] * t_ar)


def test_reused_experts_reduce_to_threshold():
    """Every token predicts only the root's experts: |E_i \\ U| = 0 throughout,
    so T_exp drops out and the same threshold rule holds with C^draft."""
    rng = np.random.default_rng(2)
    for trial in range(20):
        n = int(rng.integers(1, 30))
        parent, q, eid, c, r = random_tree(rng, n, 4, 16, 3, dyadic=True)
        c[:] = 0.5
        eid[:] = r[None]  # same experts as the root
        res = run(batch1(parent, q, eid, c, r), 16, 4.0, 1000.0)
        p = np.array([path_product(parent, q, i) for i in range(n)])
        want = sorted([i for i in range(n) if p[i] * 4.0 / 0.5 >= 1.0], key=lambda i: (-p[i], i))
        m = int(res["n_admit"][0])
        assert list(res["order"][0, :m]) == want
        assert (res["n_new"][0, :m] == 0).all()
        assert res["n_pairs"][0] == len(pair_ids(r, 16))


@pytest.mark.parametrize("m", [0, 1, 3, 6])
def test_chain_closed_form(m):
    """A chain with q = 1/2 everywhere, T_exp = 0, c = 1, T_AR = 2^m: p_i =
    2^-(i+1), so exactly the first m nodes have U_i = 2^(m-i-1) >= 1."""
    n = 10
    parent = np.arange(-1, n - 1, dtype=np.int32)
    q = np.full(n, 0.5, dtype=np.float32)
    eid = np.zeros((n, 1, 1), dtype=np.int32)
    c = np.ones(n, dtype=np.float32)
    res = run(batch1(parent, q, eid, c, None), 1, float(2 ** m), 0.0)
    assert res["n_admit"][0] == m
    assert list(res["order"][0, :m]) == list(range(m))
    np.testing.assert_array_equal(res["util"][0, :m], [2.0 ** (m - i - 1) for i in range(m)])


def test_new_experts_cost_closed_form():
    """Root children only, disjoint expert sets of sizes s_i, no root experts:
    each U_i = q_i T_AR / (s_i T_exp + c) stays fixed, so the greedy selects
    by falling U_i and keeps U_i >= 1."""
    rng = np.random.default_rng(3)
    n, L, E = 12, 2, 64
    parent = np.full(n, -1, dtype=np.int32)
    q = DYADIC[rng.integers(0, 8, n)]
    sizes = rng.integers(0, 6, n)
    eid = np.full((n, L, 6), -1, dtype=np.int32)
    nxt = 0
    for i in range(n):  # sizes[i] distinct experts in layer 1, none shared
        eid[i, 1, :sizes[i]] = np.arange(nxt, nxt + sizes[i])
        nxt += sizes[i]
    c = np.full(n, 2.0, dtype=np.float32)
    t_ar, t_exp = 16.0, 4.0
    u = q.astype(np.float64) * t_ar / (sizes * t_exp + 2.0)
    want = sorted([i for i in range(n) if u[i] >= 1.0], key=lambda i: (-u[i], i))
    res = run(batch1(parent, q, eid, c, None), E, t_ar, t_exp)
    m = int(res["n_admit"][0])
    assert list(res["order"][0, :m]) == want
    assert list(res["n_new"][0, :m]) == list(sizes[want])


def test_scaling_laws():
    """U_i = B_i / C_i is invariant when T_AR, T_exp and C^draft scale together
    (by 2^s: exact), and scaling T_AR alone by 2 keeps the selection order and
    only moves the stopping point later (utilities double exactly)."""
    rng = np.random.default_rng(4)
    for trial in range(20):
        n = int(rng.integers(2, 40))
        parent, q, eid, c, r = random_tree(rng, n, 3, 12, 3)
        base = run(batch1(parent, q, eid, c, r), 12, 6.0, 0.75)
        sc = run(batch1(parent, q, eid, (c * 8).astype(np.float32), r), 12, 48.0, 6.0)
        for key in ("order", "util", "n_new", "n_admit", "n_pairs"):
            np.testing.assert_array_equal(base[key], sc[key])
        dbl = run(batch1(parent, q, eid, c, r), 12, 12.0, 0.75)
        m = int(base["n_admit"][0])
        assert dbl["n_admit"][0] >= m
        # every utility doubles, so the argmax at each step is unchanged
        # while the base run goes on
        np.testing.assert_array_equal(dbl["order"][0, :m], base["order"][0, :m])
        np.testing.assert_array_equal(dbl["util"][0, :m], 2 * base["util"][0, :m])


def test_max_admit_is_a_prefix():
    rng = np.random.default_rng(5)
    for trial in range(20):
        n = int(rng.integers(2, 40))
        parent, q, eid, c, r = random_tree(rng, n, 3, 12, 3)
        full = run(batch1(parent, q, eid, c, r), 12, 20.0, 0.5)
        m = int(full["n_admit"][0])
        for cap in range(1, m + 2):
            part = run(batch1(parent, q, eid, c, r), 12, 20.0, 0.5, max_admit=cap)
            mm = min(cap, m)
            assert part["n_admit"][0] == mm
            np.testing.assert_array_equal(part["order"][0, :mm], full["order"][0, :mm])
            np.testing.assert_array_equal(part["util"][0, :mm], full["util"][0, :mm])


def test_invariant_to_id_order_duplicates_and_expert_relabeling():
    rng = np.random.default_rng(6)
    for trial in range(10):
        n = int(rng.integers(2, 30))
        parent, q, eid, c, r = random_tree(rng, n, 4, 10, 3)
        base = run(batch1(parent, q, eid, c, r), 10, 20.0, 0.5)
        perm_rows = eid[..., rng.permutation(3)]
        dup = np.concatenate([perm_rows, perm_rows[..., :1], np.full((n, 4, 1), -1)], axis=-1)
        rdup = np.concatenate([r, r[:, :1], np.full((4, 1), 12)], axis=-1)
        relabel = np.stack([rng.permutation(10) for _ in range(4)])  # per layer
        def rl(a):
            out = a.copy()
            for l in range(4):
                ok = (a[..., l, :] >= 0) & (a[..., l, :] < 10)
                out[..., l, :] = np.where(ok, relabel[l][np.clip(a[..., l, :], 0, 9)], a[..., l, :])
            return out
        for e2, r2 in ((dup.astype(np.int32), rdup.astype(np.int32)), (rl(eid), rl(r))):
            o = run(batch1(parent, q, e2, c, r2), 10, 20.0, 0.5)
            for key in ("order", "util", "n_new", "n_admit", "n_pairs"):
                np.testing.assert_array_equal(base[key], o[key])


def _frontier(parent, admitted, valid_nodes):
    return [i for i in valid_nodes if not admitted[i] and (parent[i] < 0 or admitted[parent[i]])]


@pytest.mark.parametrize("wl_name", sorted(TREE_WORKLOADS))
def test_greedy_invariants_on_synthetic_trees(wl_name):
    """On the synthetic workloads: the selection is closed under parents;
    every selected U_i >= 1; the n_new values telescope to the final union
    size; at each step the selected node is the largest utility on the
    frontier (ties: lower index); and when the selection stops every
    frontier node has U_i < 1.  Sets, products and utilities are recomputed
    here with numpy."""
    wl = TREE_WORKLOADS[wl_name]
    d = make_trees(wl, 4, seed=11)
    res = X.expand(d["parent"], d["q"], d["eid"], d["c_draft"], wl.n_experts, wl.t_ar,
                   wl.t_exp, d["root_eid"], d["n_nodes"])
    for t in range(4):
        n = int(d["n_nodes"][t])
        parent, q, eid = d["parent"][t, :n], d["q"][t, :n], d["eid"][t, :n]
        c = d["c_draft"][t, :n]
        sets = [pair_ids(eid[i], wl.n_experts) for i in range(n)]
        union = pair_ids(d["root_eid"][t], wl.n_experts)
        u0 = len(union)
        p = np.array([path_product(parent, q, i) for i in range(n)])
        admitted = np.zeros(n, dtype=bool)
        m = int(res["n_admit"][t])
        assert res["status"][t] == 0

        def util(i):
            nn = len(np.setdiff1d(sets[i], union))
            return p[i] * wl.t_ar / (nn * wl.t_exp + float(c[i])), nn

        for s in range(m):
            j = int(res["order"][t, s])
            front = _frontier(parent, admitted, range(n))
            assert j in front
            uj, nj = util(j)
            np.testing.assert_allclose(res["util"][t, s], uj, rtol=1e-12)
            assert res["n_new"][t, s] == nj and res["util"][t, s] >= 1.0
            for i in front:
                ui, _ = util(i)
                assert ui <= uj * (1 + 1e-12) or (abs(ui - uj) <= 1e-12 * uj and i > j)
            admitted[j] = True
            union = np.union1d(union, sets[j])
        assert res["n_pairs"][t] == len(union)
        assert int(res["n_new"][t, :m].sum()) == len(union) - u0
        for i in _frontier(parent, admitted, range(n)):
            assert util(i)[0] < 1.0


def test_invalid_inputs_set_status_and_clamp_counts():
    parent = np.array([[-1, -1, 0, 1]], dtype=np.int32)
    q = np.array([[0.5, np.nan, 0.5, 0.5]], dtype=np.float32)
    eid = np.zeros((1, 4, 1, 1), dtype=np.int32)
    c = np.array([[1, 1, np.inf, 1]], dtype=np.float32)
    r = X.expand(parent, q, eid, c, 2, 8.0, 1.0, None, np.array([4]))
    assert r["status"][0] == X.ST_BAD_CONF | X.ST_BAD_DRAFT_COST
    assert list(r["order"][0, :r["n_admit"][0]]) == [0]  # 2 has bad C^draft, 3 hangs below 1
    r = X.expand(parent, q, eid, c, 2, 8.0, 1.0, None, np.array([7]))
    assert r["status"][0] & X.ST_BAD_COUNT
    r = X.expand(parent, q, eid, c, 2, 8.0, 1.0, None, np.array([-3]))
    assert r["status"][0] == X.ST_BAD_COUNT and r["n_admit"][0] == 0
    r = X.expand(parent, q, eid, c, 2, 8.0, 1.0, None, np.array([0]))
    assert r["status"][0] == 0 and r["n_admit"][0] == 0 and r["n_pairs"][0] == 0


def test_zero_benefit_admits_nothing():
    rng = np.random.default_rng(7)
    parent, q, eid, c, r = random_tree(rng, 20, 2, 8, 2)
    res = run(batch1(parent, q, eid, c, r), 8, 0.0, 1.0)
    assert res["n_admit"][0] == 0
    assert res["n_pairs"][0] == len(pair_ids(r, 8))
