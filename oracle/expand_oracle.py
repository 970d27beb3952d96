"""Plain CPU oracle of routing-aware adaptive speculative expansion.

TEST INFRASTRUCTURE.  Only the test-suite, the smoke check and the benchmark's
CPU-baseline leg use this module.  It shares no code with the HIP library and
neither imports the other; both consume the arrays of `synth`.

What it computes (Sec. "Routing-aware Adaptive Speculative Expansion"):

  prefix confidence  p_i = product of the draft confidences on the path from
                     the first draft token down to token i ("Expected
                     Benefit"), taken root-down: p_i = p_parent(i) * q_i;
  expected benefit   B_i = p_i * T_AR;
  marginal cost      dC_i = |E_i \\ U| * T_exp, with U the union of the
                     predicted experts of the tokens already selected (Eq.
                     for the marginal verification cost);
  total cost         C_i = dC_i + C_i^draft;
  utility            U_i = B_i / C_i (Eq. for the utility), admitted
                     greedily while the best candidate has U_i >= 1.

Readings where the paper leaves a choice (each is fixed here):
  * Candidates form a tree whose root is the last verified token; node i is a
    candidate once its parent is selected (or it hangs off the root), since a
    token is accepted only after all of its prefix is.
  * Greedy means best-first: each step takes the candidate of largest U_i
    (ties: smallest node index) and recomputes the set difference against
    the grown union; it stops when the best U_i < 1, when no candidate is
    left, or after `max_admit` selections (max_admit <= 0: no limit).
  * E_i is a set of (layer, expert) pairs: the k experts each MoE layer is
    predicted to activate for token i, summed over layers, so T_exp is the
    cost of one more expert at one layer.  Expert ids outside [0, E) are
    padding and ignored; repeated ids count once.
  * The union starts from the root token's experts (it is verified in any
    case) when they are given, else empty.
  * C_i^draft is an input per node; it must be finite and positive.
  * Nodes with an invalid parent (not -1 and not an earlier node), a draft
    confidence outside [0, 1] or an invalid C^draft are never selected, and
    neither is anything below them; status bits report them (1, 2, 4), and
    bit 8 a node count outside [0, N] (then clamped).

Arithmetic: fp64, in the order B_i = p_i * T_AR, C_i = n_i * T_exp + C_i^draft,
U_i = B_i / C_i, without fused multiply-adds (Python floats).  Draft
confidences and C^draft are stored as float32 and upcast exactly.
"""

from __future__ import annotations

import numpy as np

ST_BAD_PARENT = 1
ST_BAD_CONF = 2
ST_BAD_DRAFT_COST = 4
ST_BAD_COUNT = 8


def expert_pairs(eid_rows, n_experts: int) -> set:
    """E_i as the set of (layer, expert) pairs of one token; eid_rows is
    [L][k] (ids outside [0, E) ignored)."""
    out = set()
    for layer, row in enumerate(eid_rows):
        for e in row:
            e = int(e)
            if 0 <= e < n_experts:
                out.add((layer, e))
    return out


def expand_tree(parent, q, eid, c_draft, n_experts: int, t_ar: float, t_exp: float,
                root_eid=None, max_admit: int = 0) -> dict:
    """Greedy selection on one draft tree of n = len(parent) nodes.

    parent[i]   index of the parent node, -1 for a child of the root
    q[i]        draft confidence of token i given its prefix (float32)
    eid[i]      [L][k] predicted expert ids of token i
    c_draft[i]  C_i^draft (float32)
    root_eid    [L][k] expert ids of the root token, or None

    Returns the selected nodes in selection order with U_i and |E_i \\ U| at
    their selection, the final union size and the status bits.
    """
    n = len(parent)
    status = 0
    valid = [True] * n
    for i in range(n):
        pa = int(parent[i])
        if not (pa == -1 or 0 <= pa < i):
            valid[i] = False
            status |= ST_BAD_PARENT
        qi = float(np.float32(q[i]))
        if not (0.0 <= qi <= 1.0):
            valid[i] = False
            status |= ST_BAD_CONF
        ci = float(np.float32(c_draft[i]))
        if not (ci > 0.0 and ci < float("inf")):
            valid[i] = False
            status |= ST_BAD_DRAFT_COST

    # prefix confidence, root-down (a parent always precedes its children)
    p = [None] * n
    for i in range(n):
        if not valid[i]:
            continue
        pa = int(parent[i])
        base = 1.0 if pa < 0 else p[pa]
        if base is None:
            continue  # below an invalid node: never a candidate
        p[i] = base * float(np.float32(q[i]))

    sets = [expert_pairs(eid[i], n_experts) for i in range(n)]
    union = expert_pairs(root_eid, n_experts) if root_eid is not None else set()

    admitted = [False] * n
    order, util, n_new = [], [], []
    while max_admit <= 0 or len(order) < max_admit:
        best, best_u, best_n = -1, 0.0, 0
        for i in range(n):
            if admitted[i] or p[i] is None:
                continue
            pa = int(parent[i])
            if pa >= 0 and not admitted[pa]:
                continue
            n_i = len(sets[i] - union)
            benefit = p[i] * t_ar
            cost = float(n_i) * t_exp + float(np.float32(c_draft[i]))
            u = benefit / cost
            if best < 0 or u > best_u:
                best, best_u, best_n = i, u, n_i
        if best < 0 or not (best_u >= 1.0):
            break
        admitted[best] = True
        union |= sets[best]
        order.append(best)
        util.append(best_u)
        n_new.append(best_n)
    return {"order": order, "util": util, "n_new": n_new,
            "n_pairs": len(union), "status": status}


def expand(parent, q, eid, c_draft, n_experts: int, t_ar: float, t_exp: float,
           root_eid=None, n_nodes=None, max_admit: int = 0) -> dict:
    """Batch of T trees in the padded layout of the library call.

    parent [T][N] int32, q [T][N] float32, eid [T][N][L][k] int32,
    c_draft [T][N] float32, root_eid [T][L][k] int32 or None,
    n_nodes [T] int32 or None (all N).

    Returns order [T][N] (selected node ids in selection order, -1 after),
    util [T][N] float64 (0 after), n_new [T][N] int32 (0 after), and per tree
    n_admit, n_pairs and status.
    """
    parent = np.asarray(parent)
    T, N = parent.shape
    order = np.full((T, N), -1, dtype=np.int32)
    util = np.zeros((T, N), dtype=np.float64)
    n_new = np.zeros((T, N), dtype=np.int32)
    n_admit = np.zeros(T, dtype=np.int32)
    n_pairs = np.zeros(T, dtype=np.int32)
    status = np.zeros(T, dtype=np.int32)
    for t in range(T):
        n = N if n_nodes is None else int(n_nodes[t])
        st = 0
        if n < 0 or n > N:
            st |= ST_BAD_COUNT
            n = min(max(n, 0), N)
        r = expand_tree(parent[t, :n], q[t, :n], eid[t, :n], c_draft[t, :n], n_experts,
                        t_ar, t_exp, None if root_eid is None else root_eid[t], max_admit)
        m = len(r["order"])
        order[t, :m] = r["order"]
        util[t, :m] = r["util"]
        n_new[t, :m] = r["n_new"]
        n_admit[t] = m
        n_pairs[t] = r["n_pairs"]
        status[t] = st | r["status"]
    return {"order": order, "util": util, "n_new": n_new, "n_admit": n_admit,
            "n_pairs": n_pairs, "status": status}
