"""The pins catch plausible mistakes in the oracle.

Each case plants one mistake in a private copy of the oracle's source (on the
CPU, in memory; the oracle file is never touched), loads the copy as its own
module and runs the brute-force gating comparison of test_oracle_pins over
every seed, flag set and confidence mode.  A mistake that no comparison
detects fails the test.  The mistakes cover each step of Sec. "Reuse-aware
Expert Gating": the clamp of negative confidences inside g ("Cross-token
expert importance aggregation"), the ranking and candidate set of TopCap
("Global preferred expert selection"), the sign, size and target of the bias
and the source of the gate weights ("Soft routing bias for reuse promotion").
A second set plants mistakes in the expert FFN, the int4 dequantisation and
the combine (the MoE layer's definition) and runs every pin of those steps; a
third, in the router, the plain top-k and its gap, the tie rule and the
bucketing.
"""

import itertools
import os
import types

import pytest

from tests.test_oracle_pins import (GATE_FLAGS, W_MODES, check_ffn_pins, check_gate_case,
                                    check_route_and_bucket_pins)

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


# Mistakes in the expert FFN (SwiGLU of the gate and up projections, then the
# down projection), the int4 group dequantisation and the combine.
FFN_MUTATIONS = [
    ("gate_up_swapped",
     "silu(X @ Wg.T) * (X @ Wu.T)",
     "silu(X @ Wu.T) * (X @ Wg.T)"),
    ("down_not_transposed",
     "(X @ Wu.T)) @ Wd.T",
     "(X @ Wu.T)) @ Wd"),
    ("sigmoid_for_silu",
     "return z / (1.0 + np.exp(-z))",
     "return 1.0 / (1.0 + np.exp(-z))"),
    ("token_rows_mod_k",
     "toks = rows // k",
     "toks = rows % k"),
    ("shared_rows_shifted",
     "out[B * k + s * B: B * k + (s + 1) * B]",
     "out[B * k + s: B * k + s + B]"),
    ("int4_zero_point_7",
     "(q - 8.0)",
     "(q - 7.0)"),
    ("int4_nibbles_swapped",
     "q[:, 0::2] = codes & 0x0F\n    q[:, 1::2] = codes >> 4",
     "q[:, 0::2] = codes >> 4\n    q[:, 1::2] = codes & 0x0F"),
    ("int4_scales_tiled",
     "np.repeat(s, 32, axis=1)",
     "np.tile(s, (1, 32))"),
    ("combine_weights_reversed",
     "gw[b, j] * eo[b * k + j]",
     "gw[b, k - 1 - j] * eo[b * k + j]"),
    ("combine_shared_dropped",
     "acc = acc + eo[B * k + s * B + b]",
     "acc = acc + 0.0 * eo[B * k + s * B + b]"),
    ("combine_slots_token_minor",
     "eo[b * k + j]",
     "eo[j * B + b]"),
    ("combine_shared_token_major",
     "eo[B * k + s * B + b]",
     "eo[B * k + b * n_shared + s]"),
]


@pytest.mark.parametrize("name,old,new", FFN_MUTATIONS, ids=[m[0] for m in FFN_MUTATIONS])
def test_ffn_pins_catch_mutation(name, old, new):
    mod = _mutant(name, old, new)
    try:
        check_ffn_pins(mod)
    except (AssertionError, ValueError, IndexError):
        return
    pytest.fail(f"mutation {name} passes every pin of the FFN, dequantisation and combine")


def test_unmutated_copy_passes_ffn_pins():
    check_ffn_pins(_mutant("none", "import numpy as np", "import numpy as np"))


# Mistakes in the router, the plain top-k and its gap ("Soft routing bias for
# reuse promotion" uses the top-1 minus (k+1)-th gap), the tie rule and the
# bucketing.
ROUTE_MUTATIONS = [
    ("gap_to_kth",
     "logits[b, o[0]] - logits[b, o[k]]",
     "logits[b, o[0]] - logits[b, o[k - 1]]"),
    ("gap_sign",
     "logits[b, o[0]] - logits[b, o[k]]",
     "logits[b, o[k]] - logits[b, o[0]]"),
    ("plain_idx_in_value_order",
     "plain_idx[b] = np.sort(o[:k])",
     "plain_idx[b] = o[:k]"),
    ("ties_toward_higher_index",
     "np.lexsort((np.arange(v.size), -v))",
     "np.lexsort((-np.arange(v.size), -v))"),
    ("bf16_shift_15",
     "<< np.uint32(16)",
     "<< np.uint32(15)"),
    ("router_rows_as_columns",
     "logits = X @ W.T",
     "logits = X @ W.reshape(W.shape[1], W.shape[0])"),
    ("bucket_slots_reversed",
     "for a in range(n):\n        e = flat[a]\n        slot[fill[e]] = a",
     "for a in reversed(range(n)):\n        e = flat[a]\n        slot[fill[e]] = a"),
    ("offset_shifted",
     "fill = offset[:E].copy()",
     "fill = offset[1:].copy() - 1"),
    ("uniq_not_compacted",
     "uniq[n_uniq] = e",
     "uniq[e] = e"),
    ("reuse_ratio_inverted",
     "n_uniq / n if n else 0.0",
     "n / n_uniq if n_uniq else 0.0"),
]


@pytest.mark.parametrize("name,old,new", ROUTE_MUTATIONS, ids=[m[0] for m in ROUTE_MUTATIONS])
def test_route_and_bucket_pins_catch_mutation(name, old, new):
    mod = _mutant(name, old, new)
    try:
        check_route_and_bucket_pins(mod)
    except (AssertionError, ValueError, IndexError):
        return
    pytest.fail(f"mutation {name} passes every pin of routing and bucketing")


def test_unmutated_copy_passes_route_and_bucket_pins():
    check_route_and_bucket_pins(_mutant("none", "import numpy as np", "import numpy as np"))
