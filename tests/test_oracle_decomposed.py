"""Pins for oracle.decomposed: by brute force every decomposed path equals
the dense definition (itself pinned to torch float64 and finite differences),
softmax rows recovered from the pieces sum to 1, the merge is independent of
task order, null rows are skipped, and the max-shifted merge survives scores
that overflow the literal Num/Den form in fp32 (App. A.1)."""
import numpy as np
import pytest

from oracle import decomposed, dense, planner


def _inputs(seed, B, L, H, d, scale=1.0):
    rng = np.random.default_rng(seed)
    return [scale * rng.standard_normal((B, L, H, d)) for _ in range(4)]


CASES = [(c, N, itr) for c, Ns, depths in ((7, (7, 23, 64, 100), (0, 1, 2, 3)), (13, (40,), (1, 2)))
         for N in Ns for itr in depths]


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("c,N,itr", CASES)
def test_merged_forward_equals_dense(c, N, itr, causal):
    Q, K, V, _ = _inputs(N * 10 + itr, 2, N, 2, 8)
    tasks = planner.build_tasks(N, c, itr, planner.PAPER_INTEREST_SETS[c])
    O, LSE = decomposed.merged_forward(Q, K, V, tasks, causal)
    Od, LSEd = dense.attention_forward(Q, K, V, causal)
    np.testing.assert_allclose(O, Od, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(LSE, LSEd, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("N,itr", [(23, 1), (64, 2), (100, 1), (50, 3)])
def test_numden_and_globallse_backward_equal_dense(N, itr, causal):
    Q, K, V, dO = _inputs(N + itr, 1, N, 2, 8)
    tasks = planner.build_tasks(N, 7, itr, (0, 1, 3))
    dQ, dK, dV, O, LSE = dense.attention_backward(Q, K, V, dO, causal)
    On, _, _ = decomposed.numden_forward(Q, K, V, tasks, causal)
    np.testing.assert_allclose(On, O, rtol=1e-12, atol=1e-13)
    for got in (decomposed.numden_backward(Q, K, V, dO, tasks, causal),
                decomposed.globallse_backward(Q, K, V, dO, O, LSE, tasks, causal)):
        for g, w in zip(got, (dQ, dK, dV)):
            np.testing.assert_allclose(g, w, rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_row_mass_is_one(causal):
    Q, K, V, _ = _inputs(7, 1, 80, 2, 8)
    for itr in (1, 2):
        tasks = planner.build_tasks(80, 7, itr, (0, 1, 3))
        _, LSE = dense.attention_forward(Q, K, V, causal)
        mass = decomposed.row_mass(Q, K, tasks, LSE, causal)
        np.testing.assert_allclose(mass, 1.0, atol=2e-15 * 80)


def test_merge_is_order_independent():
    Q, K, V, _ = _inputs(8, 1, 60, 2, 8)
    tasks = planner.build_tasks(60, 7, 2, (0, 1, 3))
    O0, L0 = decomposed.merged_forward(Q, K, V, tasks, True)
    rng = np.random.default_rng(9)
    for _ in range(3):
        order = rng.permutation(len(tasks))
        O1, L1 = decomposed.merged_forward(Q, K, V, tasks, True, order=order)
        np.testing.assert_allclose(O1, O0, rtol=1e-13, atol=1e-14)
        np.testing.assert_allclose(L1, L0, rtol=1e-13, atol=1e-14)


def test_null_rows_exist_and_are_skipped():
    """A causal task can keep no key for some rows (e.g. task 4 = chunks
    (0,4,5): chunk 0 is not its owner and every later key is causal-masked)."""
    N = 70
    Q, K, V, _ = _inputs(10, 1, N, 1, 8)
    task = planner.build_tasks(N, 7, 1, (0, 1, 3))[4]
    acc, ell, m = decomposed.task_statistics(Q, K, V, task, causal=True)
    null = ~np.isfinite(m[0, 0])
    assert null.sum() == 10 and (task["tokens"][null] < 10).all()
    assert (ell[0, 0, null] == 0).all() and (acc[0, null] == 0).all()
    # merged first, those null rows meet an empty accumulator; the null
    # contribution must leave it empty and the result still equal dense
    tasks = planner.build_tasks(N, 7, 1, (0, 1, 3))
    O, LSE = decomposed.merged_forward(Q, K, V, tasks, True, order=[4, 0, 1, 2, 3, 5, 6])
    Od, LSEd = dense.attention_forward(Q, K, V, True)
    np.testing.assert_allclose(O, Od, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(LSE, LSEd, rtol=1e-12, atol=1e-13)


def test_overflow_numden_fp32_vs_max_shift():
    """Scores with lse > ln(FLT_MAX) ~ 88.72 (App. A.1): the literal Num/Den
    form in fp32 goes non-finite, the max-shifted merge stays exact."""
    N = 49
    Q, K, V, _ = _inputs(11, 1, N, 1, 16)
    K = Q * 12.0                                   # q.k/sqrt(d) of order 12^2
    Q = Q * 12.0
    tasks = planner.build_tasks(N, 7, 1, (0, 1, 3))
    Od, LSEd = dense.attention_forward(Q, K, V, causal=False)
    assert LSEd.max() > 88.72
    O32, _, _ = decomposed.numden_forward(Q, K, V, tasks, False, dtype=np.float32)
    assert not np.isfinite(O32).all()
    O, LSE = decomposed.merged_forward(Q, K, V, tasks, False)
    assert np.isfinite(O).all()
    np.testing.assert_allclose(O, Od, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(LSE, LSEd, rtol=1e-13)
