"""The kernels' tile decisions as the plan predicts them (App. A.2).

cqsa_plan_fwd_tile_decisions counts, per (32-query wave, 64-key tile) pair
that a work group visits, whether the block summaries call it masked for the
wave, clear or mixed (the inner forward and the dQ kernel, at their
work-group heights); cqsa_plan_bwd_tile_decisions adds the dK/dV kernel's
(32-key group, query tile of 64 or 32 rows) decisions.  The GPU tests
require the kernels' own counters to equal these counts.  Here the planner's
counts are pinned on the CPU:

* against the same rules applied to the oracle planner's tasks;
* the rules are sound with respect to the paper's pair mask: every pair a
  skipped tile (for the work group or the wave) holds is masked, every pair of
  a clear tile is kept, and no kept pair lies outside the visited tiles;
* closed forms for the undecomposed call.
"""
import numpy as np
import pytest

import paper_2604_20819_amd as cq
from oracle import planner as oplan

BLOCK = 64


def rule_counts(tasks, causal, rows, exact_check=False):
    """The kernel's decision rules over the oracle's tasks (one batch element
    and head).  With exact_check, also verifies each verdict against the
    task's dense pair mask."""
    out = [0, 0, 0]
    for task in tasks:
        bits = task["bits"]
        L = len(bits)
        bor, band = oplan.block_summaries(bits, BLOCK)
        nkt = (L + BLOCK - 1) // BLOCK
        keep = oplan.local_mask(task, causal) if exact_check else None
        for first in range(0, L, rows):
            last = min(L, first + rows) - 1
            qand = np.uint32(0xFFFFFFFF)
            for b in range(first // BLOCK, last // BLOCK + 1):
                qand &= band[b]
            visited = [k for k in range(nkt)
                       if not (causal and k * BLOCK > last) and (qand & band[k]) == 0]
            if exact_check:
                # tiles the work group skips hold no kept pair of its queries
                for k in set(range(nkt)) - set(visited):
                    assert not keep[first:last + 1, k * BLOCK:(k + 1) * BLOCK].any()
            for q0 in range(first, last + 1, 32):
                q1 = min(q0 + 31, L - 1)
                wor, wand = bor[q0 // BLOCK], band[q0 // BLOCK]
                for k in visited:
                    k0, k1 = k * BLOCK, min(k * BLOCK + BLOCK - 1, L - 1)
                    if (wand & band[k]) != 0 or (causal and k0 > q1):
                        v = 0
                    elif (wor & bor[k]) == 0 and (not causal or k1 <= q0) and k0 + BLOCK <= L:
                        v = 1
                    else:
                        v = 2
                    out[v] += 1
                    if exact_check:
                        sub = keep[q0:q1 + 1, k0:k1 + 1]
                        if v == 0:
                            assert not sub.any(), (q0, k)
                        if v == 1:
                            assert sub.all() and sub.shape == (q1 - q0 + 1, BLOCK), (q0, k)
    return tuple(out)


def kv_rule_counts(tasks, causal, rows, qtile, exact_check=False):
    """The dK/dV kernel's rules: key strips of `rows`, 32-key groups, query
    tiles of `qtile` rows (64 or 32) whose summaries are those of block
    q * qtile // 64."""
    per_block = BLOCK // qtile
    out = [0, 0, 0]
    for task in tasks:
        bits = task["bits"]
        L = len(bits)
        bor, band = oplan.block_summaries(bits, BLOCK)
        nqt = (L + qtile - 1) // qtile
        keep = oplan.local_mask(task, causal) if exact_check else None
        for first in range(0, L, rows):
            last = min(L, first + rows) - 1
            kand = np.uint32(0xFFFFFFFF)
            for b in range(first // BLOCK, last // BLOCK + 1):
                kand &= band[b]
            visited = [q for q in range(nqt)
                       if not (causal and q * qtile + qtile - 1 < first)
                       and (kand & band[q // per_block]) == 0]
            if exact_check:
                for q in set(range(nqt)) - set(visited):
                    assert not keep[q * qtile:q * qtile + qtile, first:last + 1].any()
            for k0 in range(first, last + 1, 32):
                k1 = min(k0 + 31, L - 1)
                wor, wand = bor[k0 // BLOCK], band[k0 // BLOCK]
                for q in visited:
                    q0 = qtile * q
                    if (wand & band[q // per_block]) != 0 or (causal and q0 + qtile - 1 < k0):
                        v = 0
                    elif (wor & bor[q // per_block]) == 0 and (not causal or q0 >= k1):
                        v = 1
                    else:
                        v = 2
                    out[v] += 1
                    if exact_check:
                        sub = keep[q0:min(q0 + qtile, L), k0:k1 + 1]
                        if v == 0:
                            assert not sub.any(), (q0, k0)
                        if v == 1:
                            assert sub.all(), (q0, k0)
    return tuple(out)


def fwd_rows(d):
    return 256 if 96 <= d <= 192 else 128


def dq_rows(d):
    return 256 if 96 <= d <= 160 else 128


def kv_rows(d):
    return 256 if d in (96, 128) else 128


def kv_qtile(d):
    return 64 if d == 96 else 32


@pytest.mark.parametrize("N,itr,causal,d", [(700, 1, False, 128), (700, 1, True, 64),
                                            (1500, 2, True, 128), (1000, 2, False, 256),
                                            (3000, 1, True, 96), (130, 1, True, 128)])
def test_rules_are_sound_and_match_the_planner(N, itr, causal, d):
    tasks = oplan.build_tasks(N, 7, itr, (0, 1, 3))
    want = rule_counts(tasks, causal, fwd_rows(d), exact_check=True)
    for B, H in ((1, 1), (2, 3)):
        p = cq.cqsa_plan(N, H, d, causal, 0, cq.make_opts(B=B, depth=itr))
        assert p.fwd_tile_decisions() == tuple(B * H * x for x in want)
    assert want[1] + want[2] > 0


@pytest.mark.parametrize("levels,N,causal", [([(13, (0, 1, 3, 9)), (7, (0, 1, 3))], 2600, False),
                                             ([(21, (0, 1, 4, 14, 16))], 5000, True)])
def test_other_interest_sets(levels, N, causal):
    depth = len(levels)
    tasks = oplan.build_tasks_levels(N, levels)
    want = rule_counts(tasks, causal, 256)
    p = cq.cqsa_plan(N, 2, 128, causal, 0, cq.make_opts(depth=depth, levels=levels))
    assert p.fwd_tile_decisions() == tuple(2 * x for x in want)


def test_undecomposed_closed_forms():
    # non-causal, no group bits: nothing masked; every wave sees all tiles,
    # the ragged last one mixed
    L, d = 3000, 128
    p = cq.cqsa_plan(L, 1, d, False, 0, cq.make_opts(depth=0))
    waves, tiles = -(-L // 32), -(-L // 64)
    assert p.fwd_tile_decisions() == (0, waves * (tiles - 1), waves)
    # causal, L a multiple of the work-group rows: work group s visits the
    # tiles up to its last query; for a wave, the tiles wholly at or below
    # its first query are clear, the one holding its queries (the diagonal)
    # mixed, the later ones masked
    L, rows = 2048, 256
    p = cq.cqsa_plan(L, 1, 128, True, 0, cq.make_opts(depth=0))
    m = c = x = 0
    for s in range(L // rows):
        visited = (s + 1) * rows // 64
        for q0 in range(s * rows, (s + 1) * rows, 32):
            q1 = q0 + 31
            for k in range(visited):
                if 64 * k > q1:
                    m += 1
                elif 64 * k + 63 <= q0:
                    c += 1
                else:
                    x += 1
    assert p.fwd_tile_decisions() == (m, c, x)
    # one diagonal tile per wave, and every wave sees its work group's tiles
    assert x == L // 32
    assert m + c + x == sum((s + 1) * rows // 64 * rows // 32 for s in range(L // rows))


@pytest.mark.parametrize("N,itr,causal,d", [(700, 1, False, 128), (700, 1, True, 64),
                                            (1500, 2, True, 96), (1000, 2, False, 256),
                                            (3000, 1, True, 160), (130, 1, True, 128)])
def test_backward_rules_are_sound_and_match_the_planner(N, itr, causal, d):
    tasks = oplan.build_tasks(N, 7, itr, (0, 1, 3))
    want_q = rule_counts(tasks, causal, dq_rows(d), exact_check=True)
    want_k = kv_rule_counts(tasks, causal, kv_rows(d), kv_qtile(d), exact_check=True)
    for B, H in ((1, 1), (2, 3)):
        p = cq.cqsa_plan(N, H, d, causal, 0, cq.make_opts(B=B, depth=itr, with_backward=True))
        dq, kv = p.bwd_tile_decisions()
        assert dq == tuple(B * H * x for x in want_q)
        assert kv == tuple(B * H * x for x in want_k)
    assert want_k[1] + want_k[2] > 0


def test_fp32_plans_are_not_counted():
    p = cq.cqsa_plan(500, 1, 64, False, 0, cq.make_opts(dtype="f32", depth=1))
    for f in (p.fwd_tile_decisions, p.bwd_tile_decisions):
        with pytest.raises(cq.CqsaError) as e:
            f()
        assert e.value.status == -2


def test_kv_query_tile_rows():
    for d in range(32, 257, 32):
        assert cq.cqsa_bwd_kv_query_tile(d) == kv_qtile(d)
    for d in (0, 16, 48, 100, 288, -32):
        assert cq.cqsa_bwd_kv_query_tile(d) == 0
