"""Reader of tests/golden/expand_worked_examples.txt (hand-derived trees)."""

from __future__ import annotations

import os
from dataclasses import dataclass, field
from fractions import Fraction

import numpy as np

PATH = os.path.join(os.path.dirname(__file__), "golden", "expand_worked_examples.txt")


@dataclass
class WorkedTree:
    name: str
    E: int
    L: int
    K: int
    t_ar: float
    t_exp: float
    max_admit: int = 0
    root: list | None = None
    nodes: list = field(default_factory=list)  # (parent, q, c, [L][K] ids)
    expect: dict = field(default_factory=dict)

    def arrays(self, n_pad: int | None = None):
        """Padded single-tree batch: parent [1][N], q [1][N] f32, eid
        [1][N][L][K], c_draft [1][N] f32, root_eid [1][L][K] or None,
        n_nodes [1]."""
        n = len(self.nodes)
        N = n if n_pad is None else n_pad
        parent = np.full((1, N), -1, dtype=np.int32)
        q = np.zeros((1, N), dtype=np.float32)
        c = np.ones((1, N), dtype=np.float32)
        eid = np.full((1, N, self.L, self.K), -1, dtype=np.int32)
        for i, (pa, qi, ci, ids) in enumerate(self.nodes):
            parent[0, i], q[0, i], c[0, i] = pa, qi, ci
            eid[0, i] = ids
        root = None if self.root is None else np.asarray(self.root, dtype=np.int32)[None]
        return parent, q, eid, c, root, np.array([n], dtype=np.int32)


def _layers(tokens, L, K):
    groups = " ".join(tokens).split("|")
    rows = [[int(v) for v in g.split()] for g in groups]
    assert len(rows) == L and all(len(r) == K for r in rows), (tokens, L, K)
    return rows


def load() -> list[WorkedTree]:
    trees, cur = [], None
    with open(PATH) as f:
        for raw in f:
            line = raw.split("#", 1)[0].strip()
            if not line:
                continue
            tok = line.split()
            if tok[0] == "tree":
                cur = WorkedTree(tok[1], 0, 0, 0, 0.0, 0.0)
            elif tok[0] == "shape":
                kv = dict(zip(tok[1::2], tok[2::2]))
                cur.E, cur.L, cur.K = int(kv["E"]), int(kv["L"]), int(kv["K"])
                cur.t_ar, cur.t_exp = float(kv["T_AR"]), float(kv["T_EXP"])
                cur.max_admit = int(kv.get("MAX", 0))
            elif tok[0] == "root":
                cur.root = _layers(tok[1:], cur.L, cur.K)
            elif tok[0] == "node":
                assert int(tok[1]) == len(cur.nodes)
                kv = dict(zip(tok[2:8:2], tok[3:8:2]))
                assert tok[8] == "eids"
                cur.nodes.append((int(kv["parent"]), float(kv["q"]), float(kv["c"]),
                                  _layers(tok[9:], cur.L, cur.K)))
            elif tok[0] == "expect":
                key, vals = tok[1], tok[2:]
                if key == "util":
                    cur.expect[key] = [float(Fraction(v)) for v in vals]
                elif key in ("n_pairs", "status"):
                    cur.expect[key] = int(vals[0])
                else:
                    cur.expect[key] = [int(v) for v in vals]
            elif tok[0] == "end":
                trees.append(cur)
                cur = None
            else:
                raise ValueError(f"bad line: {raw!r}")
    return trees
