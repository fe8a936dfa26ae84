"""Pins for oracle.planner against what the paper prints: the interest-set
table (App. C), the worked examples of Sections 3.1 and 3.3, exactly-once
coverage by brute force, and the tile census of App. A.2."""
import numpy as np
import pytest

from oracle import planner
from tests.conftest import golden_path


def _golden_sets():
    sets, pairs = {}, []
    for line in open(golden_path("interest_sets.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        if line.startswith("pair"):
            lhs, rhs = line[len("pair"):].split("->")
            lhs = [int(x) for x in lhs.split()]
            pairs.append((lhs[0], tuple(lhs[1:]), tuple(int(x) for x in rhs.split())))
            continue
        parts = line.split()
        c, l = int(parts[0]), int(parts[1])
        sets[c] = (l, None if parts[2] == "None" else tuple(int(x) for x in parts[2:]))
    return sets, pairs


def test_interest_set_table():
    sets, pairs = _golden_sets()
    for c, (l, I) in sets.items():
        assert c == l * (l - 1) + 1
        if I is None:
            assert c not in planner.PAPER_INTEREST_SETS
            continue
        assert len(I) == l
        assert planner.PAPER_INTEREST_SETS[c] == I
        assert planner.is_perfect_difference_set(I, c)
    for c, I, P in pairs:
        assert planner.paired_interest_set(I, c) == P
        assert planner.is_perfect_difference_set(P, c)
    # non-examples: repeated differences
    assert not planner.is_perfect_difference_set((0, 1, 2), 7)
    assert not planner.is_perfect_difference_set((0, 1, 3, 4), 13)


def test_paired_sets_of_table_are_difference_sets():
    for c, I in planner.PAPER_INTEREST_SETS.items():
        assert planner.is_perfect_difference_set(planner.paired_interest_set(I, c), c)


def _golden_examples():
    out = {}
    for line in open(golden_path("worked_examples.txt")):
        line = line.strip()
        if line and not line.startswith("#"):
            key, *vals = line.split()
            out[key] = [int(v) for v in vals if v != ":"]
    return out


def test_worked_example_diag_pair():
    ex = _golden_examples()
    tasks = planner.build_tasks(7, 7, 1, (0, 1, 3))
    holding = [t for t, task in enumerate(tasks) if 0 in task["tokens"]]
    assert holding == ex["diag_pair_tasks"][1:]
    keeping = [t for t in holding
               if planner.local_mask(tasks[t], False)[list(tasks[t]["tokens"]).index(0)][list(tasks[t]["tokens"]).index(0)]]
    assert keeping == [0]


def test_task0_keeps_only_own_diagonal():
    ex = _golden_examples()
    N = 70
    task = planner.build_tasks(N, 7, 1, (0, 1, 3))[0]
    keep = planner.local_mask(task, False)
    chunk = task["tokens"] // 10
    kept_diag = sorted({int(chunk[a]) for a in range(len(chunk)) for b in range(len(chunk))
                        if chunk[a] == chunk[b] and keep[a, b]})
    assert kept_diag == ex["task0_kept_diagonal"]
    # every off-diagonal chunk pair of the task is kept entirely
    off = chunk[:, None] != chunk[None, :]
    assert keep[off].all()


def test_n49_example():
    ex = _golden_examples()
    t1 = planner.build_tasks(49, 7, 1, (0, 1, 3))
    assert len(t1) == 7 and all(len(t["tokens"]) == ex["n49_depth1_len"][0] for t in t1)
    s, e = planner.balanced_chunk_layout(ex["n49_depth1_len"][0], 7)
    assert set((e - s).tolist()) == {ex["n49_depth2_chunk"][0]}
    t2 = planner.build_tasks(49, 7, 2, (0, 1, 3))
    assert len(t2) == 49 and all(len(t["tokens"]) == ex["n49_depth2_len"][0] for t in t2)


def test_balanced_layout():
    s, e = planner.balanced_chunk_layout(23, 7)
    assert (e - s).tolist() == [4, 4, 3, 3, 3, 3, 3]
    assert s[0] == 0 and e[-1] == 23 and (s[1:] == e[:-1]).all()


@pytest.mark.parametrize("c", [7, 13])
@pytest.mark.parametrize("causal", [False, True])
def test_exactly_once_coverage(c, causal):
    I = planner.PAPER_INTEREST_SETS[c]
    Ns = [7, 49, 50, 64, 100] if c == 7 else [13, 40, 90]
    depths = [1, 2, 3] if c == 7 else [1, 2]
    for N in Ns:
        for itr in depths:
            tasks = planner.build_tasks(N, c, itr, I)
            assert len(tasks) == c ** itr
            counts = planner.coverage_counts(tasks, N, causal)
            want = np.tril(np.ones((N, N), dtype=np.int64)) if causal else np.ones((N, N), dtype=np.int64)
            assert (counts == want).all(), (N, itr)


# Section 3.3: a different valid interest set may be used at each depth.
MIXED_LEVELS = [
    [(7, (0, 1, 3)), (13, (0, 1, 3, 9))],
    [(13, (0, 1, 3, 9)), (7, (0, 1, 3))],
    [(3, (0, 1)), (7, (0, 1, 3)), (3, (0, 1))],
    [(21, (0, 1, 4, 14, 16)), (3, (0, 1))],
]


@pytest.mark.parametrize("levels", MIXED_LEVELS, ids=lambda v: "-".join(str(c) for c, _ in v))
@pytest.mark.parametrize("causal", [False, True])
def test_mixed_levels_cover_every_pair_once(levels, causal):
    """Brute force: with a set per level every kept pair is computed by exactly
    one task, there are prod(c_t) tasks, and each token sits in prod(l_t)."""
    ntask = int(np.prod([c for c, _ in levels]))
    per_token = int(np.prod([len(I) for _, I in levels]))
    for N in (ntask // 2 + 1, ntask, 2 * ntask + 5, 150):
        tasks = planner.build_tasks_levels(N, levels)
        assert len(tasks) == ntask
        appear = np.zeros(N, dtype=np.int64)
        for t in tasks:
            assert (np.diff(t["tokens"]) > 0).all()
            appear[t["tokens"]] += 1
        assert (appear == per_token).all(), N
        counts = planner.coverage_counts(tasks, N, causal)
        want = np.tril(np.ones((N, N), dtype=np.int64)) if causal else np.ones((N, N), dtype=np.int64)
        assert (counts == want).all(), N


def test_mixed_levels_bits_are_disjoint_per_level():
    """Level t's groups use bits [s_t, s_t + l_t - 1), disjoint across levels."""
    levels = [(7, (0, 1, 3)), (13, (0, 1, 3, 9))]
    for task in planner.build_tasks_levels(200, levels):
        assert {b for b, _ in task["groups"]} == set(range(2 + 3))
        level2 = task["bits"] >> np.uint32(2)
        assert (level2 < 8).all()
        assert (np.bitwise_count(level2) <= 1).all() and (np.bitwise_count(task["bits"] & 3) <= 1).all()


def test_each_chunk_in_l_tasks_and_tokens_ascending():
    for itr in (1, 2):
        tasks = planner.build_tasks(100, 7, itr, (0, 1, 3))
        appear = np.zeros(100, dtype=np.int64)
        for t in tasks:
            g = t["tokens"]
            assert (np.diff(g) > 0).all()
            appear[g] += 1
        assert (appear == 3 ** itr).all()


def test_runs_reassemble_tokens_and_bits():
    for N, itr in ((1000, 1), (1000, 2), (343, 3)):
        for task in planner.build_tasks(N, 7, itr, (0, 1, 3)):
            rs = planner.runs(task)
            assert len(rs) <= 3 ** itr
            g = np.concatenate([np.arange(s, s + n) for s, n, _ in rs])
            b = np.concatenate([np.full(n, bits, dtype=np.uint32) for _, n, bits in rs])
            assert (g == task["tokens"]).all() and (b == task["bits"]).all()


def test_bits_per_level():
    """Each token holds at most one bit per level; the owner chunk none."""
    for task in planner.build_tasks(343, 7, 3, (0, 1, 3)):
        for t in range(3):
            level = (task["bits"] >> (2 * t)) & 3
            assert (level != 3).all()


def _golden_census():
    census, mixed = {}, {}
    for line in open(golden_path("tile_census.txt")):
        p = line.split()
        if not p or p[0].startswith("#"):
            continue
        if p[0] == "census":
            census[(int(p[1]), int(p[2]))] = tuple(float(x) for x in p[3:6])
        elif p[0] == "mixed":
            mixed[(int(p[1]), int(p[2]))] = (float(p[3]), int(p[4]), float(p[5]))
    return census, mixed


def test_tile_census_65536():
    census, _ = _golden_census()
    for (N, itr), (full, clear, mix) in census.items():
        f, c, m, tot = planner.tile_census(planner.build_tasks(N, 7, itr, (0, 1, 3)))
        assert f + c + m == tot
        assert round(100 * f / tot, 1) == full
        assert round(100 * c / tot, 1) == clear
        assert round(100 * m / tot, 2) == mix


@pytest.mark.slow
def test_mixed_fraction_and_bound():
    _, mixed = _golden_census()
    for (N, itr), (mix, nb, bound) in mixed.items():
        tasks = planner.build_tasks(N, 7, itr, (0, 1, 3))
        Li = max(len(t["tokens"]) for t in tasks)
        assert -(-Li // 128) == nb
        assert round(100 * 3 / nb, 2) == bound
        f, c, m, tot = planner.tile_census(tasks)
        assert round(100 * m / tot, 2) == mix
        assert 100 * m / tot <= bound
