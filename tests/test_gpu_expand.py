"""GPU parity of routing-aware adaptive expansion: s2moe_expand through the
C ABI against the expansion oracle.  Every output is compared exactly: the
selection, counts and status are integers, and the utilities are the same
fp64 operations in the same order on both sides (no fused multiply-add,
correctly rounded division)."""

import numpy as np
import pytest

from oracle import expand_oracle as X
from synth.trees import TREE_WORKLOADS, make_trees
from tests.expand_fixtures import load
from tests.gpu_helpers import log

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

KEYS = ("order", "util", "n_new", "n_admit", "n_pairs", "status")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_15018_amd as s2
    s2.load()


def run_gpu(parent, q, eid, c, root, n_nodes, E, t_ar, t_exp, max_admit=0):
    import paper_2608_15018_amd as s2
    T, N = parent.shape
    dev = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    out = s2.ExpandOut(T, N)
    s2.expand(dev(parent), dev(q), dev(eid), dev(c), dev(n_nodes), out, E, t_ar, t_exp,
              root_eid=dev(root), max_admit=max_admit)
    torch.cuda.synchronize()
    return out.host()


def compare(got, ref, label, trees=None):
    sel = slice(None) if trees is None else trees
    for k in KEYS:
        g, r = got[k][sel], ref[k]
        if not np.array_equal(g, r):
            bad = np.argwhere(g != r)[:5]
            raise AssertionError(f"{label}: {k} differs at {bad.tolist()}: "
                                 f"gpu {g[tuple(bad[0])]} oracle {r[tuple(bad[0])]}")


def both(label, parent, q, eid, c, root, n_nodes, E, t_ar, t_exp, max_admit=0):
    log(f"[expand] {label}: T={parent.shape[0]} N={parent.shape[1]} L={eid.shape[2]} "
        f"k={eid.shape[3]} E={E} max_admit={max_admit}")
    got = run_gpu(parent, q, eid, c, root, n_nodes, E, t_ar, t_exp, max_admit)
    ref = X.expand(parent, q, eid, c, E, t_ar, t_exp, root, n_nodes, max_admit)
    compare(got, ref, label)
    return got


def test_worked_examples_on_gpu():
    for tree in load():
        for pad in (0, 7, 300):
            a = list(tree.arrays(n_pad=len(tree.nodes) + pad))
            a[0][0, len(tree.nodes):] = 5  # garbage in the padding
            got = both(f"worked {tree.name} pad {pad}", *a, tree.E, tree.t_ar, tree.t_exp,
                       tree.max_admit)
            m = int(got["n_admit"][0])
            assert list(got["order"][0, :m]) == tree.expect["order"]
            assert list(got["util"][0, :m]) == tree.expect["util"]


@pytest.mark.parametrize("wl_name", sorted(TREE_WORKLOADS))
def test_synthetic_model_trees(wl_name):
    wl = TREE_WORKLOADS[wl_name]
    d = make_trees(wl, 24, seed=3)
    both(wl_name, d["parent"], d["q"], d["eid"], d["c_draft"], d["root_eid"], d["n_nodes"],
         wl.n_experts, wl.t_ar, wl.t_exp)
    # cheaper drafts admit more and exercise longer greedy runs
    both(wl_name + " cheap", d["parent"], d["q"], d["eid"], d["c_draft"] / 16, d["root_eid"],
         d["n_nodes"], wl.n_experts, wl.t_ar * 4, wl.t_exp)


def random_batch(rng, T, N, L, E, k, ragged=True, dup_ids=True, bad=0.0):
    parent = np.full((T, N), -1, dtype=np.int32)
    for t in range(T):
        for i in range(1, N):
            parent[t, i] = rng.integers(-1, i)
    q = rng.random((T, N)).astype(np.float32) ** 0.3
    lo = -1 if dup_ids else 0
    eid = rng.integers(lo, E + (1 if dup_ids else 0), size=(T, N, L, k)).astype(np.int32)
    c = (rng.random((T, N)) * 0.5 + 0.05).astype(np.float32)
    root = rng.integers(0, E, size=(T, L, k)).astype(np.int32)
    n_nodes = (rng.integers(0, N + 1, T) if ragged else np.full(T, N)).astype(np.int32)
    if bad:
        m = rng.random((T, N)) < bad
        parent[m & (rng.random((T, N)) < 0.5)] = N + 3
        q[m & (rng.random((T, N)) < 0.5)] = np.nan
        c[m & (rng.random((T, N)) < 0.5)] = 0.0
    return parent, q, eid, c, root, n_nodes


@pytest.mark.parametrize("T,N,L,E,k", [
    (5, 1, 1, 1, 1), (6, 33, 3, 7, 2), (4, 97, 5, 40, 3), (3, 256, 4, 64, 4),
    (3, 257, 4, 32, 2), (2, 511, 2, 33, 5), (2, 700, 2, 16, 3), (2, 1024, 2, 8, 2),
    (3, 64, 7, 1024, 1), (2, 16, 128, 8, 32),
    (3, 200, 6, 128, 5), (2, 300, 3, 255, 3), (2, 64, 9, 250, 7), (3, 120, 48, 128, 8),
])
def test_random_trees_across_tilings(T, N, L, E, k):
    """Random tree shapes (any earlier node as parent), padding and repeated
    ids, ragged node counts including 0 and N; N spans 1, 2 and 4 nodes per
    thread and E spans 1..1024 (k 5-8 at E 128-255 too, ids unaligned with
    16-byte chunks when L k is odd)."""
    rng = np.random.default_rng(T * 1000 + N)
    a = random_batch(rng, T, N, L, E, k)
    t_exp = 0.5 / max(1, L * k)
    both(f"random {N}", *a, E, 2.0, t_exp)
    both(f"random {N} capped", *a, E, 2.0, t_exp, max_admit=3)


def test_no_root_zero_cost_and_zero_benefit():
    rng = np.random.default_rng(9)
    p, q, e, c, r, n = random_batch(rng, 4, 80, 3, 16, 2)
    both("no root", p, q, e, c, None, n, 16, 3.0, 0.05)
    both("T_exp 0", p, q, e, c, r, n, 16, 3.0, 0.0)
    both("T_AR 0", p, q, e, c, r, n, 16, 0.0, 0.05)


def test_invalid_nodes_and_counts():
    rng = np.random.default_rng(10)
    p, q, e, c, r, n = random_batch(rng, 6, 60, 2, 8, 2, bad=0.1)
    n[0], n[1] = -2, 61  # clamped, status bit 8
    got = both("invalid", p, q, e, c, r, n, 8, 4.0, 0.05)
    assert got["status"][0] & 8 and got["status"][1] & 8


def test_large_batch_and_determinism():
    """Many trees of the Qwen3-shaped workload: sampled trees against the
    oracle, and two launches give identical bits."""
    wl = TREE_WORKLOADS["t_qwen3"]
    T = 512
    d = make_trees(wl, T, seed=21)
    args = (d["parent"], d["q"], d["eid"], d["c_draft"], d["root_eid"], d["n_nodes"])
    log(f"[expand] large: T={T} N={wl.max_nodes}")
    g1 = run_gpu(*args, wl.n_experts, wl.t_ar, wl.t_exp)
    g2 = run_gpu(*args, wl.n_experts, wl.t_ar, wl.t_exp)
    for k in KEYS:
        assert np.array_equal(g1[k], g2[k]), k
    pick = np.array([0, 1, 2, 100, 255, 256, 400, T - 1])
    ref = X.expand(*(a[pick] for a in args[:4]), wl.n_experts, wl.t_ar, wl.t_exp,
                   args[4][pick], args[5][pick])
    compare({k: v[pick] for k, v in g1.items()}, ref, "large sampled")


def test_max_nodes_bound():
    import paper_2608_15018_amd as s2
    for L, E, k in ((48, 128, 8), (26, 64, 6), (128, 1024, 32)):
        m = s2.expand_max_nodes(L, E, k)
        log(f"[expand] max_nodes L={L} E={E} k={k}: {m}")
        if m == 0 or m == 1024:
            continue
        rng = np.random.default_rng(0)
        both(f"at max_nodes {m}", *random_batch(rng, 1, m, L, E, k, ragged=False), E, 2.0, 0.01)
        a = random_batch(rng, 1, m + 1, L, E, k)
        with pytest.raises(s2.S2moeError, match="LDS"):
            run_gpu(*a, E, 2.0, 0.01)
    assert s2.expand_max_nodes(48, 128, 8) >= 116  # the Qwen3-shaped trees fit
