"""GPU tests of the kernels' tile decisions (App. A.2).

With tile counting on, every wave of the inner forward (and of the backward's
dQ kernel, and every 32-key group of its dK/dV kernel) adds the decisions it
took over the tiles its work group visited: masked for the wave (skipped),
clear (no mask work) or mixed (per-pair tests).  The counts must equal what
the plan's block summaries predict (cqsa_plan_fwd_tile_decisions,
cqsa_plan_bwd_tile_decisions, pinned on the CPU in
tests/test_tile_decisions.py) exactly: this checks that the kernels' window
scans, next-tile probes and tile rings visit exactly the live tiles, once
each, and decide them as the summaries say.  Counting leaves the outputs
unchanged (same bits as an uncounted call).
"""
import pytest
import torch

import paper_2604_20819_amd as cq
from paper_2604_20819_amd import synth
from tests.gpu_util import need_gpu, say

pytestmark = pytest.mark.gpu

CASES = [
    # dt, B, L, H, d, causal, depth, levels, read_in_place, tasks_per_slot
    ("bf16", 2, 3000, 3, 128, False, 1, None, None, 0),
    ("f16", 1, 5000, 2, 64, True, 2, None, None, 0),
    ("bf16", 1, 2049, 2, 256, True, 1, None, None, 0),
    ("bf16", 1, 4096, 2, 96, True, 0, None, None, 0),
    ("bf16", 1, 2600, 2, 128, False, 2, [(13, (0, 1, 3, 9)), (7, (0, 1, 3))], False, 0),
    ("bf16", 1, 777, 1, 160, True, 1, None, None, 1),
    ("f16", 1, 32768, 2, 128, True, 1, None, None, 0),
    ("bf16", 1, 9000, 2, 192, False, 2, None, False, 0),
]


def forward(plan, q, k, v, B, L, H, d):
    O = torch.empty((B, L, H, d), dtype=torch.float32, device="cuda")
    LSE = torch.empty((B, H, L), dtype=torch.float32, device="cuda")
    cq.cqsa_forward(plan, q, k, v, O, LSE)
    torch.cuda.synchronize()
    return O.cpu(), LSE.cpu(), cq.cqsa_last_stats()


@pytest.mark.parametrize("dt,B,L,H,d,causal,depth,levels,rip,tps", CASES,
                         ids=["-".join(str(x) for x in c[:7]) for c in CASES])
def test_kernel_decisions_equal_the_plan(dt, B, L, H, d, causal, depth, levels, rip, tps):
    need_gpu()
    say(f"tile counts {dt} B={B} L={L} H={H} d={d} causal={causal} depth={depth} "
        f"levels={levels} read_in_place={rip} tasks_per_slot={tps}")
    Q, K, V = synth.make_inputs(9100 + L + d, B, L, H, d, dt)
    q, k, v = (x.cuda() for x in (Q, K, V))
    plan = cq.cqsa_plan(L, H, d, causal, 0, cq.make_opts(B=B, dtype=dt, depth=depth, levels=levels,
                                                         read_in_place=rip, tasks_per_slot=tps))
    want = plan.fwd_tile_decisions()
    O0, L0, st0 = forward(plan, q, k, v, B, L, H, d)
    assert (st0["kernel_tiles_masked"], st0["kernel_tiles_clear"], st0["kernel_tiles_mixed"]) == (-1, -1, -1)
    cq.cqsa_set_tile_counting(True)
    try:
        O1, L1, st1 = forward(plan, q, k, v, B, L, H, d)
        O2, L2, st2 = forward(plan, q, k, v, B, L, H, d)
    finally:
        cq.cqsa_set_tile_counting(False)
    got = (st1["kernel_tiles_masked"], st1["kernel_tiles_clear"], st1["kernel_tiles_mixed"])
    say(f"  {plan.num_tasks} tasks, {st1['inner_launches']} launches: kernel {got}, plan {want}")
    assert got == want
    # the counters start from zero on every call
    assert (st2["kernel_tiles_masked"], st2["kernel_tiles_clear"], st2["kernel_tiles_mixed"]) == want
    assert torch.equal(O0, O1) and torch.equal(L0, L1) and torch.equal(O0, O2)
    if depth > 0:
        assert want[0] > 0 and want[2] > 0


BWD_CASES = [
    # dt, B, L, H, d, causal, depth, opts
    ("bf16", 2, 3000, 3, 128, False, 1, {}),
    ("bf16", 1, 2049, 2, 128, True, 1, dict(bwd_tasks_per_launch=1)),
    ("f16", 1, 5000, 2, 64, True, 2, {}),
    ("bf16", 1, 1500, 2, 96, True, 0, {}),
    ("bf16", 1, 2600, 2, 160, False, 1, dict(read_in_place=False)),
    ("bf16", 1, 900, 1, 256, True, 1, dict(inputs_on_device=False, acc_on_device=False)),
    ("f16", 1, 32768, 2, 128, True, 1, {}),
]


@pytest.mark.parametrize("dt,B,L,H,d,causal,depth,kw", BWD_CASES,
                         ids=["-".join(str(x) for x in c[:7]) for c in BWD_CASES])
def test_backward_kernel_decisions_equal_the_plan(dt, B, L, H, d, causal, depth, kw):
    need_gpu()
    say(f"backward tile counts {dt} B={B} L={L} H={H} d={d} causal={causal} depth={depth} {kw}")
    host = kw.get("inputs_on_device", True) is False
    Q, K, V, dO = synth.make_inputs(9200 + L + d, B, L, H, d, dt, with_dO=True, pin_memory=host)
    dev = (lambda x: x) if host else (lambda x: x.cuda())
    q, k, v, do = (dev(x) for x in (Q, K, V, dO))
    mk = ((lambda *sh: torch.empty(sh, dtype=torch.float32, pin_memory=True)) if host else
          (lambda *sh: torch.empty(sh, dtype=torch.float32, device="cuda")))
    plan = cq.cqsa_plan(L, H, d, causal, 0, cq.make_opts(B=B, dtype=dt, depth=depth, with_backward=True, **kw))
    want_q, want_k = plan.bwd_tile_decisions()
    O, LSE = mk(B, L, H, d), mk(B, H, L)
    cq.cqsa_forward(plan, q, k, v, O, LSE)
    outs = []
    for counting in (False, True):
        g = [mk(B, L, H, d) for _ in range(3)]
        cq.cqsa_set_tile_counting(counting)
        try:
            cq.cqsa_backward(plan, q, k, v, O, LSE, do, *g)
            torch.cuda.synchronize()
            st = cq.cqsa_last_stats()
        finally:
            cq.cqsa_set_tile_counting(False)
        outs.append([x.cpu() for x in g])
        got_q = (st["kernel_tiles_masked"], st["kernel_tiles_clear"], st["kernel_tiles_mixed"])
        got_k = (st["kernel_kv_tiles_masked"], st["kernel_kv_tiles_clear"], st["kernel_kv_tiles_mixed"])
        if not counting:
            assert got_q == (-1, -1, -1) and got_k == (-1, -1, -1)
    say(f"  {plan.num_tasks} tasks, {st['inner_launches']} launches: dQ {got_q} (plan {want_q}), "
        f"dK/dV {got_k} (plan {want_k})")
    assert got_q == want_q
    assert got_k == want_k
    for a, b in zip(*outs):
        assert torch.equal(a, b)
    if depth > 0:
        assert want_q[0] > 0 and want_k[0] > 0 and want_k[2] > 0


def test_fp32_and_noalloc_calls_are_not_counted():
    need_gpu()
    B, L, H, d = 1, 600, 2, 64
    Q, K, V = synth.make_inputs(9101, B, L, H, d, "f32")
    q, k, v = (x.cuda() for x in (Q, K, V))
    plan = cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(B=B, dtype="f32", depth=1))
    plan16 = cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(B=B, dtype="bf16", depth=1))
    q16, k16, v16 = (x.to(torch.bfloat16) for x in (q, k, v))
    O = torch.empty((B, L, H, d), dtype=torch.float32, device="cuda")
    LSE = torch.empty((B, H, L), dtype=torch.float32, device="cuda")
    cq.cqsa_set_tile_counting(True)
    try:
        _, _, st = forward(plan, q, k, v, B, L, H, d)
        cq.cqsa_forward_noalloc(plan16, q16, k16, v16, O, LSE)
        torch.cuda.synchronize()
        st_na = cq.cqsa_last_stats()
    finally:
        cq.cqsa_set_tile_counting(False)
    for s in (st, st_na):
        assert (s["kernel_tiles_masked"], s["kernel_tiles_clear"], s["kernel_tiles_mixed"]) == (-1, -1, -1)
