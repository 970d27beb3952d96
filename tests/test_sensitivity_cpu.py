"""Host logic of the cap x alpha reuse sweep (paper_2608_15018_amd.sensitivity):
grid, reuse ratio, deviation and the paper's improvement figure, pinned by
hand-made selections and the paper's expert-reuse table."""

import os

import numpy as np
import pytest

from paper_2608_15018_amd import sensitivity as S


def test_cap_grid_spans_k_to_3k_with_paper_value():
    assert S.caps_for(6, 16, 64) == [6, 9, 12, 15, 16, 18]
    assert S.caps_for(8, 18, 64) == [8, 12, 16, 18, 20, 24]
    assert S.caps_for(8, 14, 20) == [8, 12, 14, 16, 20]  # capped at E


def test_reuse_ratio_and_deviation_by_hand():
    idx = np.array([[0, 1], [1, 2], [0, 1]])
    assert S.reuse_ratio(idx, 2) == 3 / 6
    plain = np.array([[0, 1], [1, 3], [2, 4]])
    # token 1 lost 3 (gained 2), token 2 lost both: 3 of 6 slots moved
    assert S.deviation(idx, plain) == 3 / 6
    assert S.deviation(plain, plain) == 0.0


def test_improvement_matches_paper_table():
    """The paper's "Reuse Improvement" column is the relative reduction."""
    path = os.path.join(os.path.dirname(__file__), "golden", "expert_reuse.txt")
    rows = [l.split() for l in open(path) if l.strip() and not l.startswith("#")]
    for name, r0, r1, pct in rows:
        assert 100 * S.improvement(float(r0), float(r1)) == pytest.approx(float(pct), abs=0.01)


def test_summarize_means_over_batches():
    caps, alphas = [2, 3], (0.0, 1.0)
    plain = np.array([[0, 1], [2, 3]])
    s1 = {"plain_idx": plain, "idx": {(2, 0.0): plain, (3, 0.0): plain,
                                      (2, 1.0): np.array([[0, 1], [0, 1]]),
                                      (3, 1.0): np.array([[0, 1], [1, 3]])}}
    s2 = {"plain_idx": plain, "idx": {k: plain for k in s1["idx"]}}
    out = S.summarize(2, [s1, s2], caps, alphas)
    assert out["plain_reuse_ratio"] == 1.0
    g = out["grid"]["2/1.0"]
    assert g["reuse_ratio"] == (0.5 + 1.0) / 2 and g["improvement"] == 0.25
    assert g["deviation"] == (0.5 + 0.0) / 2
    g = out["grid"]["3/1.0"]
    assert g["reuse_ratio"] == (0.75 + 1.0) / 2 and g["deviation"] == (0.25 + 0.0) / 2
    md = S.to_markdown([dict(out, shape="x", B=2, rho=0.0, batches=2, caps=caps,
                             alphas=list(alphas), k=2, paper_cap=3)])
    assert "| 3 (1.5k) paper |" in md
