"""GPU tests of the backward with several tasks per launch.

With inputs read in place and device-resident gradients, one dQ and one
dK/dV launch run all the tasks of a launch group; each task's rows go to its
own fp32 buffer and a gather-merge adds them into dQ, dK, dV in task order.
One task per launch instead adds each task's rows into the gradients
directly, tasks one after another on each stream.  Both add the same rounded
values (the scaled gradient is rounded before the addition) in the same
order, so every grouping must give the same bits: all tasks in one launch,
groups of three (7 tasks: 3 + 3 + 1, the later groups adding to what the
earlier ones merged), and one task per launch.  Against float64 the usual
backward bounds hold (rel-L2 <= 2e-2 and the arithmetic bound).
"""
import numpy as np
import pytest
import torch

import paper_2604_20819_amd as cq
from paper_2604_20819_amd import synth
from tests.gpu_util import need_gpu, rel_l2, say
from tests.test_gpu_backward import REL, oracle_grads

pytestmark = pytest.mark.gpu


def run(Q, K, V, dO, causal, depth, bwd_tpl, levels=None):
    B, L, H, d = Q.shape
    dt = {torch.float16: "f16", torch.bfloat16: "bf16"}[Q.dtype]
    plan = cq.cqsa_plan(L, H, d, causal, 0,
                        cq.make_opts(B=B, dtype=dt, depth=depth, with_backward=True,
                                     bwd_tasks_per_launch=bwd_tpl, levels=levels))
    q, k, v, do = (x.cuda() for x in (Q, K, V, dO))
    O = torch.empty((B, L, H, d), dtype=torch.float32, device="cuda")
    LSE = torch.empty((B, H, L), dtype=torch.float32, device="cuda")
    cq.cqsa_forward(plan, q, k, v, O, LSE)
    # NaN-filled gradients: every element must be written
    dQ, dK, dV = (torch.full((B, L, H, d), float("nan"), dtype=torch.float32, device="cuda")
                  for _ in range(3))
    cq.cqsa_set_timing(True)
    try:
        cq.cqsa_backward(plan, q, k, v, O, LSE, do, dQ, dK, dV)
        torch.cuda.synchronize()
        st = cq.cqsa_last_stats()
    finally:
        cq.cqsa_set_timing(False)
    return [t.cpu() for t in (dQ, dK, dV)], plan, st


CASES = [
    ("bf16", 1, 1000, 2, 64, False, 1, None),
    ("bf16", 2, 1500, 3, 128, True, 1, None),
    ("f16", 1, 2049, 2, 128, False, 1, None),
    ("f16", 1, 3000, 2, 64, True, 2, None),
    ("bf16", 1, 777, 2, 96, True, 1, None),
    ("bf16", 1, 2600, 2, 128, False, 2, [(13, (0, 1, 3, 9)), (7, (0, 1, 3))]),
    ("bf16", 1, 900, 1, 256, True, 1, None),
]


@pytest.mark.parametrize("dt,B,L,H,d,causal,depth,levels", CASES,
                         ids=["-".join(str(x) for x in c[:7]) for c in CASES])
def test_every_grouping_gives_the_same_bits(dt, B, L, H, d, causal, depth, levels):
    need_gpu()
    say(f"batched backward {dt} B={B} L={L} H={H} d={d} causal={causal} depth={depth} "
        f"levels={levels}")
    Q, K, V, dO = synth.make_inputs(515 + L + d, B, L, H, d, dt, with_dO=True)
    res = {}
    for tpl in (0, 3, 1):
        g, plan, st = run(Q, K, V, dO, causal, depth, tpl, levels)
        n = plan.num_tasks
        gs = plan.bwd_tasks_per_launch
        groups = -(-n // gs)
        say(f"  bwd_tasks_per_launch={tpl}: {gs} per launch, {groups} groups of {n} tasks, "
            f"launches {st['inner_launches']}, merges {st['merge_launches']}")
        if tpl == 0:
            assert gs == -(-n // -(-n // 32))  # every task up to 32, in balanced launches
        else:
            assert gs == min(tpl, n)
        assert st["inner_launches"] == 2 * (groups if gs > 1 else n)
        assert st["merge_launches"] == (groups if gs > 1 else 0)
        assert st["resident_tasks"] == (gs if gs > 1 else 0)
        res[tpl] = g
    for name, i in (("dQ", 0), ("dK", 1), ("dV", 2)):
        assert np.isfinite(res[0][i].numpy()).all(), name
        assert torch.equal(res[0][i], res[1][i]), f"{name}: all tasks vs one per launch"
        assert torch.equal(res[3][i], res[1][i]), f"{name}: groups of 3 vs one per launch"
    want = oracle_grads(Q, K, V, dO, causal)
    for name, g, w in zip(("dQ", "dK", "dV"), res[0], want):
        r = rel_l2(g.numpy(), w)
        say(f"  {name} vs float64: {r:.3e}")
        assert r <= 2e-2 and r <= REL[dt], name


def test_depth2_L32768_batched_vs_undecomposed():
    """bf16 causal B=1 H=4 d=128 L=32768 at depth 2: 49 tasks, 25 + 24 per
    launch, against the undecomposed call (rel-L2 <= 1e-3) and against one
    task per launch (same bits)."""
    need_gpu()
    B, L, H, d = 1, 32768, 4, 128
    say(f"batched backward depth 2 B={B} L={L} H={H} d={d}")
    Q, K, V, dO = synth.make_inputs(20819 + 61, B, L, H, d, "bf16", with_dO=True)
    g, plan, st = run(Q, K, V, dO, True, 2, 0)
    assert plan.num_tasks == 49 and plan.bwd_tasks_per_launch == 25
    assert st["merge_launches"] == 2
    g1, _, _ = run(Q, K, V, dO, True, 2, 1)
    g0, _, _ = run(Q, K, V, dO, True, 0, 0)
    for name, i in (("dQ", 0), ("dK", 1), ("dV", 2)):
        r = rel_l2(g[i].numpy(), g0[i].numpy())
        say(f"  {name} vs undecomposed: {r:.3e}")
        assert r <= 1e-3, name
        assert torch.equal(g[i], g1[i]), name


def test_long_launches_serialise_dq_after_dkdv():
    """bf16 B=1 H=40 d=128 L=32768, non-causal, depth 1: every dK/dV launch
    spans at least 8 rounds of the GPU's resident waves, so the dQ kernels run
    after the dK/dV kernels on the caller's stream (one task per launch too:
    55 key strips x 40 heads x 8 waves per task), where shorter launches run
    them on a second stream.  All tasks in one launch and one task per launch
    give the same bits, and both match the undecomposed call (rel-L2 <= 1e-3)."""
    need_gpu()
    B, L, H, d = 1, 32768, 40, 128
    say(f"serialised dQ launches B={B} L={L} H={H} d={d}")
    Q, K, V, dO = synth.make_inputs(20819 + 62, B, L, H, d, "bf16", with_dO=True)
    g, plan, st = run(Q, K, V, dO, False, 1, 0)
    assert plan.num_tasks == 7 and plan.bwd_tasks_per_launch == 7
    # the drivers' serial-launch threshold: 8 rounds of 256 CUs x 8 waves
    strips = -(-min(plan.task(t)["L_local"] for t in range(7)) // 256)
    assert strips == 55 and strips * B * H * 8 >= 8 * 256 * 8
    g1, _, st1 = run(Q, K, V, dO, False, 1, 1)
    assert st1["inner_launches"] == 14
    g0, _, _ = run(Q, K, V, dO, False, 0, 0)
    for name, i in (("dQ", 0), ("dK", 1), ("dV", 2)):
        assert np.isfinite(g[i].numpy()).all(), name
        assert torch.equal(g[i], g1[i]), name
        r = rel_l2(g[i].numpy(), g0[i].numpy())
        say(f"  {name} vs undecomposed: {r:.3e}")
        assert r <= 1e-3, name
