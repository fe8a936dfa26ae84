"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a copy of an oracle function (CPU only: the
function's source text is edited, compiled into the oracle module's namespace
and swapped in for the duration of the case), then runs the pin tests that
guard that function.  At least one of them must fail; otherwise the pins
would not notice that mistake in the oracle.

The mistakes are the kind the oracle could plausibly contain: a dropped
scale or correction term, an off-by-one or flipped causal test, a transposed
or wrong operand, a missing rescale in the merge, a null row not skipped, a
wrong interest-set direction, colliding group bits, a masked owner chunk,
descending chunk order, and a different remainder rule.
"""
import contextlib
import inspect
import textwrap

import pytest

from oracle import decomposed, dense, planner
from tests import test_oracle_decomposed as T_dec
from tests import test_oracle_dense as T_dense
from tests import test_oracle_planner as T_plan


@contextlib.contextmanager
def mutant(module, name, old, new):
    """Swap module.name for a copy whose source has `old` replaced by `new`."""
    fn = getattr(module, name)
    src = textwrap.dedent(inspect.getsource(fn))
    assert src.count(old) == 1, f"{name}: snippet {old!r} must occur exactly once"
    ns = dict(vars(module))
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), ns)
    setattr(module, name, ns[name])
    try:
        yield
    finally:
        setattr(module, name, fn)


def caught(checks):
    """True if any pin check fails on the mutant."""
    for check in checks:
        try:
            check()
        except Exception:  # an assertion, or the mutant breaking a check outright
            return True
    return False


FWD_PINS = [
    lambda: T_dense.test_forward_matches_torch(False, (2, 37, 3, 16)),
    lambda: T_dense.test_forward_matches_torch(True, (2, 37, 3, 16)),
    T_dense.test_zero_query_gives_mean_and_prefix_mean,
    T_dense.test_constant_value_and_single_token,
]
BWD_PINS = [
    lambda: T_dense.test_backward_matches_torch_autograd(False),
    lambda: T_dense.test_backward_matches_torch_autograd(True),
    lambda: T_dense.test_backward_finite_differences(True),
]
PLAN_PINS = [
    T_plan.test_worked_example_diag_pair,
    T_plan.test_task0_keeps_only_own_diagonal,
    T_plan.test_n49_example,
    T_plan.test_balanced_layout,
    lambda: T_plan.test_exactly_once_coverage(7, False),
    T_plan.test_each_chunk_in_l_tasks_and_tokens_ascending,
    T_plan.test_bits_per_level,
]
MIXED_PINS = [
    lambda: T_plan.test_mixed_levels_cover_every_pair_once(T_plan.MIXED_LEVELS[0], False),
    T_plan.test_mixed_levels_bits_are_disjoint_per_level,
]
DEC_PINS = [
    lambda: T_dec.test_merged_forward_equals_dense(7, 23, 1, False),
    lambda: T_dec.test_merged_forward_equals_dense(7, 64, 2, True),
    lambda: T_dec.test_numden_and_globallse_backward_equal_dense(23, 1, True),
    lambda: T_dec.test_row_mass_is_one(True),
    T_dec.test_null_rows_exist_and_are_skipped,
]

MUTANTS = [
    # dense forward
    ("fwd: scale dropped", dense, "attention_forward",
     "s = alpha * (q @ k.T)", "s = (q @ k.T)", FWD_PINS),
    ("fwd: causal diagonal dropped", dense, "attention_forward",
     "np.arange(L)[None, :] <= r[:, None]", "np.arange(L)[None, :] < r[:, None]", FWD_PINS),
    ("fwd: causal direction flipped", dense, "attention_forward",
     "np.arange(L)[None, :] <= r[:, None]", "np.arange(L)[None, :] >= r[:, None]", FWD_PINS),
    ("fwd: LSE without the max", dense, "attention_forward",
     "(m + np.log(denom))[:, 0]", "(np.log(denom))[:, 0]", FWD_PINS),
    ("fwd: rows not normalised", dense, "attention_forward",
     "(p @ v) / denom", "(p @ v)", FWD_PINS),
    # dense backward
    ("bwd: D term dropped", dense, "attention_backward",
     "ds = p * (dp - D)", "ds = p * dp", BWD_PINS),
    ("bwd: dK from K instead of Q", dense, "attention_backward",
     "alpha * (ds.T @ q)", "alpha * (ds.T @ k)", BWD_PINS),
    ("bwd: dQ without alpha", dense, "attention_backward",
     "dQ[b, :, h, :] = alpha * (ds @ k)", "dQ[b, :, h, :] = (ds @ k)", BWD_PINS),
    ("bwd: dV with P untransposed", dense, "attention_backward",
     "p.T @ do", "p @ do", BWD_PINS),
    # planner
    ("plan: interest offsets subtracted", planner, "build_tasks_levels",
     "sorted(((q + o) % c) for o in I)", "sorted(((q - o) % c) for o in I)", PLAN_PINS),
    ("plan: chunks in descending order", planner, "build_tasks_levels",
     "sorted(((q + o) % c) for o in I)", "sorted(((q + o) % c for o in I), reverse=True)",
     PLAN_PINS),
    ("plan: levels share group bits", planner, "build_tasks_levels",
     "(int(offsets[t]) + (j - 1), member)", "((j - 1), member)", PLAN_PINS),
    ("plan: every level masks with the first level's set", planner, "build_tasks_levels",
     "            c, I = levels[t]\n            for j, o in enumerate(I):",
     "            c, I = levels[0]\n            for j, o in enumerate(I):", MIXED_PINS),
    ("plan: owner chunk masked too", planner, "build_tasks_levels",
     "if j == 0:\n                    continue", "pass", PLAN_PINS),
    ("plan: remainder to the last chunks", planner, "balanced_chunk_layout",
     "(1 if u < extra else 0)", "(1 if u >= c - extra else 0)", PLAN_PINS),
    # decomposed
    ("merge: old accumulator not rescaled", decomposed, "merge_into",
     "acc[b, gq, h, :] * a_old", "acc[b, gq, h, :]", DEC_PINS),
    ("merge: null rows not skipped", decomposed, "merge_into",
     "if not np.isfinite(mi):\n                    continue", "pass", DEC_PINS),
    ("merge: l not rescaled", decomposed, "merge_into",
     "ell[b, h, gq] * a_old", "ell[b, h, gq]", DEC_PINS),
    ("forward: LSE = m + l", decomposed, "merged_forward",
     "LSE = m + np.log(ell)", "LSE = m + ell", DEC_PINS),
    ("globallse: D term dropped", decomposed, "globallse_backward",
     "ds = P * (dp - D[b, g, h][:, None])", "ds = P * dp", DEC_PINS),
    ("globallse: mask not applied to P", decomposed, "globallse_backward",
     "P = np.where(keep, np.exp(np.where(keep, s, 0.0) - _f64(LSE[b, h, g])[:, None]), 0.0)",
     "P = np.exp(s - _f64(LSE[b, h, g])[:, None])", DEC_PINS),
]


@pytest.mark.parametrize("label,module,name,old,new,pins", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(label, module, name, old, new, pins):
    with mutant(module, name, old, new):
        assert caught(pins), f"no pin noticed: {label}"


def test_unmutated_oracle_passes_the_same_pins():
    """The harness itself: the same pin lists pass on the real oracle."""
    for pins in (FWD_PINS, BWD_PINS, PLAN_PINS, MIXED_PINS, DEC_PINS):
        assert not caught(pins)
