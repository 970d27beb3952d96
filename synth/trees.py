"""Seeded synthetic draft trees for routing-aware adaptive expansion.

Only random draws and tree bookkeeping live here; the prefix confidences,
set differences, utilities and the greedy selection are computed by the HIP
library and, separately, by the oracle.

Recipe (per tree, from its own PCG64 stream keyed by (seed, tree)):
  * shape: a root (the last verified token) and `depth` levels of draft
    tokens.  The first `beam` nodes of each level (breadth-first order,
    children of a node ordered by falling confidence) are expanded, each into
    `branch` children.  With the paper's draft length 8 this is depth 8; a
    per-tree beam drawn from [beam_min, beam] makes the trees ragged.
  * draft confidences: each expanded node's most likely child has a
    confidence ~ Beta(4, 1.2) (mean 0.77: drafts are usually confident about
    their first choice), and the other children take the largest shares of
    the remaining mass split by a Dirichlet(0.3) over 31 tokens (float32).
  * predicted experts: per MoE layer a Zipf(1.1) expert popularity over a
    random expert order; the root token draws k distinct experts from it, and
    each child keeps each of its parent's experts with probability `inherit`
    and fills the rest with distinct experts drawn from the popularity
    (Gumbel top-k), so nearby tokens share experts as in the paper's
    observation of cross-token expert reuse.
  * C^draft: the same value for every node.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

T_TREE = 21  # seed-key tag of this generator


@dataclass(frozen=True)
class TreeWorkload:
    name: str
    n_layers: int     # MoE layers whose expert sets are predicted
    n_experts: int    # E
    k: int            # experts per token and layer
    depth: int = 8
    branch: int = 4
    beam: int = 4
    beam_min: int = 2
    inherit: float = 0.6
    t_ar: float = 512.0     # cost of one target decoding step, in units of T_exp
    t_exp: float = 1.0
    c_draft: float = 16.0
    description: str = ""

    @property
    def max_nodes(self) -> int:
        return self.branch + (self.depth - 1) * self.beam * self.branch


# Layer counts are those of the public model architectures; experts and k
# follow the paper's model table (Table "Model and SD configurations").
TREE_WORKLOADS = {
    "t_qwen3": TreeWorkload("t_qwen3", 48, 128, 8,
                            description="Qwen3-30B-A3B-shaped draft trees: 48 MoE layers, "
                                        "128 experts, 8 per token, depth 8, branch 4, beam 2-4"),
    "t_deepseek": TreeWorkload("t_deepseek", 26, 64, 6,
                               description="DeepSeek-V2-Lite-shaped draft trees: 26 MoE layers, "
                                           "64 experts, 6 per token, depth 8, branch 4, beam 2-4"),
    "t_olmoe": TreeWorkload("t_olmoe", 16, 64, 8,
                            description="OLMoE-shaped draft trees: 16 MoE layers, 64 experts, "
                                        "8 per token, depth 8, branch 4, beam 2-4"),
    "t_gptoss": TreeWorkload("t_gptoss", 36, 128, 4,
                             description="GPT-OSS-120B-shaped draft trees: 36 MoE layers, "
                                         "128 experts, 4 per token, depth 8, branch 4, beam 2-4"),
}


def _rng(seed: int, *key: int) -> np.random.Generator:
    ss = np.random.SeedSequence(entropy=int(seed), spawn_key=tuple(int(k) for k in key))
    return np.random.Generator(np.random.PCG64(ss))


def _popularity(rng, L, E, s=1.1):
    w = 1.0 / np.arange(1, E + 1, dtype=np.float64) ** s
    logp = np.empty((L, E))
    for l in range(L):
        logp[l, rng.permutation(E)] = np.log(w / w.sum())
    return logp


def _draw_experts(rng, logp, k, keep=None):
    """k distinct experts per layer: Gumbel top-k over log-popularity, with
    the experts in `keep` ([L][E] bool) forced in."""
    key = logp + rng.gumbel(size=logp.shape)
    if keep is not None:
        key = np.where(keep, np.inf, key)
    return np.argpartition(-key, k - 1, axis=1)[:, :k].astype(np.int32)


def make_tree(wl: TreeWorkload, seed: int, tree: int, beam: int | None = None) -> dict:
    """One tree: parent [n], q [n] f32, eid [n][L][k], root_eid [L][k]."""
    rng = _rng(seed, T_TREE, tree)
    L, E, k = wl.n_layers, wl.n_experts, wl.k
    beam = rng.integers(wl.beam_min, wl.beam + 1) if beam is None else beam
    logp = _popularity(rng, L, E)
    root_eid = _draw_experts(rng, logp, k)
    parent, q, eid = [], [], []
    level = [-1]  # the root
    for _ in range(wl.depth):
        nxt = []
        for pa in level[:beam]:
            top = rng.beta(4.0, 1.2)
            rest = np.sort(rng.dirichlet(np.full(31, 0.3)))[::-1] * (1.0 - top)
            conf = np.concatenate(([top], rest))[:wl.branch]
            base = root_eid if pa < 0 else eid[pa]
            for c in range(wl.branch):
                keep = np.zeros((L, E), dtype=bool)
                kept = rng.random((L, k)) < wl.inherit
                rows = np.nonzero(kept)[0]
                keep[rows, base[kept]] = True
                parent.append(pa)
                q.append(conf[c])
                eid.append(_draw_experts(rng, logp, k, keep))
                nxt.append(len(parent) - 1)
        level = nxt
    return {"parent": np.array(parent, dtype=np.int32),
            "q": np.array(q, dtype=np.float32),
            "eid": np.stack(eid), "root_eid": root_eid}


def make_trees(wl: TreeWorkload, T: int, seed: int, n_pad: int | None = None) -> dict:
    """Batch of T ragged trees in the padded layout of the library call:
    parent [T][N] (-1 padding), q [T][N] f32, eid [T][N][L][k] (-1 padding),
    c_draft [T][N] f32, root_eid [T][L][k], n_nodes [T]."""
    N = wl.max_nodes if n_pad is None else n_pad
    L, k = wl.n_layers, wl.k
    out = {"parent": np.full((T, N), -1, dtype=np.int32),
           "q": np.zeros((T, N), dtype=np.float32),
           "eid": np.full((T, N, L, k), -1, dtype=np.int32),
           "c_draft": np.full((T, N), wl.c_draft, dtype=np.float32),
           "root_eid": np.empty((T, L, k), dtype=np.int32),
           "n_nodes": np.zeros(T, dtype=np.int32)}
    for t in range(T):
        tr = make_tree(wl, seed, t)
        n = min(len(tr["parent"]), N)
        out["parent"][t, :n] = tr["parent"][:n]
        out["q"][t, :n] = tr["q"][:n]
        out["eid"][t, :n] = tr["eid"][:n]
        out["root_eid"][t] = tr["root_eid"]
        out["n_nodes"][t] = n
    return out
