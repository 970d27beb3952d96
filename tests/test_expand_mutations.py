"""The expansion pins catch plausible mistakes in the expansion oracle.

Each case plants one mistake in a private copy of the oracle's source (on the
CPU, in memory; the oracle file is never touched) and runs every pin of
tests/test_expand_oracle.py against that copy.  A mistake that no pin
detects fails the test.  The mistakes cover each term of the utility of Sec.
"Routing-aware Adaptive Speculative Expansion" (the expected benefit p_i T_AR,
the marginal cost |E_i minus U| T_exp, the draft cost C_i^draft), the prefix
product, the union of (layer, expert) pairs, the tree frontier, the
threshold U_i >= 1 and the tie rule.
"""

import os
import types

import pytest

import tests.test_expand_oracle as T
from synth.trees import TREE_WORKLOADS
from tests.expand_fixtures import load

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "expand_oracle.py")

# (name, text in the oracle, replacement)
MUTATIONS = [
    ("expert_cost_dropped",
     "cost = float(n_i) * t_exp + float(np.float32(c_draft[i]))",
     "cost = float(np.float32(c_draft[i]))"),
    ("draft_cost_dropped",
     "cost = float(n_i) * t_exp + float(np.float32(c_draft[i]))",
     "cost = float(n_i) * t_exp + 1e-300"),
    ("benefit_without_t_ar",
     "benefit = p[i] * t_ar",
     "benefit = p[i]"),
    ("set_difference_reversed",
     "n_i = len(sets[i] - union)",
     "n_i = len(union - sets[i])"),
    ("prefix_not_multiplied",
     "p[i] = base * float(np.float32(q[i]))",
     "p[i] = float(np.float32(q[i]))"),
    ("frontier_ignores_tree",
     "if pa >= 0 and not admitted[pa]:\n                continue",
     "if False:\n                continue"),
    ("strict_threshold",
     "if best < 0 or not (best_u >= 1.0):",
     "if best < 0 or not (best_u > 1.0):"),
    ("tie_to_larger_index",
     "if best < 0 or u > best_u:",
     "if best < 0 or u >= best_u:"),
    ("union_not_grown",
     "union |= sets[best]",
     "union = union"),
    ("root_experts_ignored",
     "union = expert_pairs(root_eid, n_experts) if root_eid is not None else set()",
     "union = set()"),
    ("padding_ids_counted",
     "if 0 <= e < n_experts:",
     "if e < n_experts:"),
    ("layers_merged",
     "out.add((layer, e))",
     "out.add((0, e))"),
    ("confidence_above_one_accepted",
     "if not (0.0 <= qi <= 1.0):",
     "if not (0.0 <= qi):"),
]


def _mutant(name, old, new):
    text = open(SRC).read()
    assert text.count(old) >= 1, f"{name}: '{old}' no longer in the oracle"
    mod = types.ModuleType(f"expand_oracle_mutant_{name}")
    exec(compile(text.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


def run_pins(mod, monkeypatch):
    """Every pin of the expansion oracle, with the oracle replaced by mod."""
    monkeypatch.setattr(T, "X", mod)
    for tree in load():
        T.test_worked_examples(tree)
    T.test_worked_examples_padded_layout_is_inert()
    T.test_zero_expert_cost_is_confidence_threshold()
    T.test_reused_experts_reduce_to_threshold()
    for m in (0, 1, 3, 6):
        T.test_chain_closed_form(m)
    T.test_new_experts_cost_closed_form()
    T.test_scaling_laws()
    T.test_max_admit_is_a_prefix()
    T.test_invariant_to_id_order_duplicates_and_expert_relabeling()
    for wl_name in sorted(TREE_WORKLOADS):
        T.test_greedy_invariants_on_synthetic_trees(wl_name)
    T.test_invalid_inputs_set_status_and_clamp_counts()
    T.test_zero_benefit_admits_nothing()


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_pins_catch_mutation(name, old, new, monkeypatch):
    mod = _mutant(name, old, new)
    try:
        run_pins(mod, monkeypatch)
    except (AssertionError, ValueError, IndexError, ZeroDivisionError):
        return
    pytest.fail(f"mutation {name} passes every pin of the expansion oracle")


def test_unmutated_copy_passes(monkeypatch):
    run_pins(_mutant("none", "import numpy as np", "import numpy as np"), monkeypatch)
