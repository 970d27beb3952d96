"""The gating pins catch plausible mistakes in the oracle.

Each case plants one mistake in a private copy of the oracle's source (on the
CPU, in memory; the oracle file is never touched), loads the copy as its own
module and runs the brute-force gating comparison of test_oracle_pins over
every seed, flag set and confidence mode.  A mistake that no comparison
detects fails the test.  The mistakes cover each step of Sec. "Reuse-aware
Expert Gating": the clamp of negative confidences inside g ("Cross-token
expert importance aggregation"), the ranking and candidate set of TopCap
("Global preferred expert selection"), the sign, size and target of the bias
and the source of the gate weights ("Soft routing bias for reuse promotion").
"""

import itertools
import os
import types

import pytest

from tests.test_oracle_pins import GATE_FLAGS, W_MODES, check_gate_case

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "s2moe_oracle.py")

# (name, text in the oracle, replacement)
MUTATIONS = [
    ("topcap_ascending_g",
     "chosen = cand[rank_order(g[cand])][:cap]",
     "chosen = cand[rank_order(-g[cand])][:cap]"),
    ("activated_only_ascending_g",
     "chosen = cand[rank_order(g[cand])][:cap]",
     "chosen = cand[rank_order(-g[cand] if flags & PREF_ACTIVATED_ONLY else g[cand])][:cap]"),
    ("unclamped_confidence_in_g",
     "g += w[b] * ell[b]",
     "g += np.asarray(conf_w, dtype=np.float64)[b] * ell[b]"),
    ("no_bias_switch_off",
     "active = bool(np.any(w > 0.0))",
     "active = True"),
    ("candidates_not_restricted",
     "if flags & PREF_ACTIVATED_ONLY:",
     "if False:"),
    ("bias_on_non_preferred",
     "if pref[e]:",
     "if not pref[e]:"),
    ("bias_negative",
     "lam = float(alpha) * np.asarray(gap, dtype=np.float64)",
     "lam = -float(alpha) * np.asarray(gap, dtype=np.float64)"),
    ("absolute_flag_ignored",
     "elif flags & BIAS_ABSOLUTE:",
     "elif False:"),
    ("gate_from_biased_ignored",
     "src = biased if flags & GATE_FROM_BIASED else ell",
     "src = ell"),
    ("gate_always_from_biased",
     "src = biased if flags & GATE_FROM_BIASED else ell",
     "src = biased"),
    ("cap_off_by_one",
     "[:cap]",
     "[:cap - 1]"),
]


def _mutant(name, old, new):
    text = open(SRC).read()
    assert text.count(old) >= 1, f"{name}: '{old}' no longer in the oracle"
    mod = types.ModuleType(f"oracle_mutant_{name}")
    exec(compile(text.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_pins_catch_mutation(name, old, new):
    mod = _mutant(name, old, new)
    for seed, flags, w_mode in itertools.product(range(30), GATE_FLAGS, W_MODES):
        try:
            check_gate_case(mod, seed, flags, w_mode)
        except (AssertionError, ValueError, IndexError):
            return
    pytest.fail(f"mutation {name} passes every brute-force gating comparison")


def test_unmutated_copy_passes():
    """The in-memory copy itself (no substitution) passes every comparison,
    so a caught mutation is the substitution's doing."""
    mod = _mutant("none", "import numpy as np", "import numpy as np")
    for seed, flags, w_mode in itertools.product(range(30), GATE_FLAGS, W_MODES):
        check_gate_case(mod, seed, flags, w_mode)
