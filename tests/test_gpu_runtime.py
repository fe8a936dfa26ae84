"""GPU tests of the runtime around the kernels: the caller-allocator hook, the
workspace cache release, ordering on a caller stream, and the per-call
statistics (bytes moved, launch counts, workspace vs the footprint model)."""
import numpy as np
import pytest
import torch

import paper_2604_20819_amd as cq
from paper_2604_20819_amd import synth
from tests.gpu_util import need_gpu, run_forward, say

pytestmark = pytest.mark.gpu


def _inputs(L=3000, H=2, d=128, dt="bf16", seed=31):
    return synth.make_inputs(seed, 1, L, H, d, dt)


def test_caller_allocator_serves_the_workspace():
    """With a caller allocator installed, every workspace byte comes from it,
    is released after the call, and the results are bit-identical to the
    built-in workspace; an allocator that fails gives DEVICE_OOM."""
    need_gpu()
    Q, K, V = _inputs()
    say("caller allocator")
    O0, L0, _ = run_forward(Q, K, V, True, depth=2)
    calls = []
    held = {}

    def alloc(n):
        t = torch.empty((n,), dtype=torch.uint8, device="cuda")
        held[t.data_ptr()] = t
        calls.append(n)
        return t.data_ptr()

    def release(ptr):
        held.pop(ptr)

    cq.cqsa_set_allocator(alloc, release)
    try:
        cq.cqsa_set_timing(True)
        O1, L1, _ = run_forward(Q, K, V, True, depth=2)
        st = cq.cqsa_last_stats()
    finally:
        cq.cqsa_set_timing(False)
        cq.cqsa_set_allocator(None, None)
    assert calls == [st["workspace_bytes"]] and not held
    assert torch.equal(O0, O1) and torch.equal(L0, L1)

    cq.cqsa_set_allocator(lambda n: 0, lambda p: None)
    try:
        with pytest.raises(cq.CqsaError) as e:
            run_forward(Q, K, V, True, depth=2)
        assert e.value.status == -4
    finally:
        cq.cqsa_set_allocator(None, None)


def test_torch_caching_allocator_helper():
    need_gpu()
    Q, K, V = _inputs(L=1500, seed=32)
    O0, L0, _ = run_forward(Q, K, V, False, depth=1)
    held = cq.use_torch_allocator()
    try:
        O1, L1, _ = run_forward(Q, K, V, False, depth=1)
    finally:
        cq.cqsa_set_allocator(None, None)
    assert not held
    assert torch.equal(O0, O1) and torch.equal(L0, L1)


def test_release_workspace_between_calls():
    need_gpu()
    Q, K, V = _inputs(L=2000, seed=33)
    O0, L0, _ = run_forward(Q, K, V, True, depth=1)
    cq.cqsa_release_workspace()
    O1, L1, _ = run_forward(Q, K, V, True, depth=1)
    cq.cqsa_release_workspace()
    assert torch.equal(O0, O1) and torch.equal(L0, L1)


def test_work_is_ordered_on_the_callers_stream():
    """Inputs produced on a side stream (default priority) and consumed there
    right after the call, with no device-wide synchronisation in between."""
    need_gpu()
    Q, K, V = _inputs(L=4000, seed=34)
    O0, L0, _ = run_forward(Q, K, V, False, depth=1)
    plan = cq.cqsa_plan(4000, 2, 128, False, 0, cq.make_opts(dtype="bf16", depth=1))
    qh, kh, vh = (x.cuda() for x in (Q, K, V))
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        # a slow producer on the side stream: the call must wait for it
        big = torch.ones(8192, 8192, device="cuda")
        for _ in range(20):
            big = big * 1.0
        q = qh + (big[:1, :1] * 0).to(qh.dtype)
        O = torch.empty((1, 4000, 2, 128), dtype=torch.float32, device="cuda")
        LSE = torch.empty((1, 2, 4000), dtype=torch.float32, device="cuda")
        cq.cqsa_forward(plan, q, kh, vh, O, LSE)
        Oc, Lc = O.clone(), LSE.clone()   # consumed on the same stream
    s.synchronize()
    assert torch.equal(Oc.cpu(), O0) and torch.equal(Lc.cpu(), L0)


@pytest.mark.parametrize("in_place", [True, False])
@pytest.mark.parametrize("depth,tps", [(1, 0), (2, 0), (1, 3)])
def test_call_statistics(depth, tps, in_place):
    """Bytes staged (none when the inputs are read in place), launch counts
    and workspace size follow the plan."""
    need_gpu()
    L, H, d = 3000, 2, 128
    Q, K, V = _inputs(L=L, H=H, d=d, seed=35)
    cq.cqsa_set_timing(True)
    try:
        O, LSE, plan = run_forward(Q, K, V, True, depth=depth, tasks_per_slot=tps,
                                   read_in_place=in_place)
        st = cq.cqsa_last_stats()
    finally:
        cq.cqsa_set_timing(False)
    rows = sum(plan.task(t)["L_local"] for t in range(plan.num_tasks))
    g = plan.tasks_per_slot
    groups = -(-plan.num_tasks // g)
    assert st["depth"] == depth and st["num_tasks"] == plan.num_tasks
    assert plan.reads_in_place == int(in_place)
    assert st["d2d_bytes"] == (0 if in_place else 3 * rows * H * d * 2)
    assert st["h2d_bytes"] == 0 and st["d2h_bytes"] == 0
    assert st["inner_launches"] == groups and st["merge_launches"] == groups
    assert 0 < st["workspace_bytes"] <= plan.modelled_device_bytes
    assert st["ms_wall"] > 0 and 0 < st["ms_inner_busy"] <= st["ms_inner"] + 1e-6
    assert np.isfinite(O.numpy()).all()


def test_back_to_back_calls_on_plans_destroyed_at_once():
    """Calls return before their GPU work runs.  Each call copies its plan's
    task tables to the device from library-owned pinned memory, so a plan may
    be destroyed as soon as the call returns: here eight forwards on fresh
    plans of two shapes (staged and in place, one and several launch groups)
    are issued back to back, each plan dropped at once, and every output must
    equal the same call made in isolation."""
    need_gpu()
    import gc
    L, H, d = 2500, 2, 64
    Q, K, V = _inputs(L=L, H=H, d=d, seed=61)
    q, k, v = (x.cuda() for x in (Q, K, V))
    shapes = [dict(depth=1, read_in_place=True), dict(depth=2, read_in_place=False, tasks_per_slot=4),
              dict(depth=2, read_in_place=True), dict(depth=1, read_in_place=False)]

    def call(kw, O, LSE):
        plan = cq.cqsa_plan(L, H, d, True, 0, cq.make_opts(**kw))
        cq.cqsa_forward(plan, q, k, v, O, LSE)
        del plan
        gc.collect()

    refs = []
    for kw in shapes:
        O = torch.empty((1, L, H, d), dtype=torch.float32, device="cuda")
        LSE = torch.empty((1, H, L), dtype=torch.float32, device="cuda")
        call(kw, O, LSE)
        torch.cuda.synchronize()
        refs.append((O.cpu(), LSE.cpu()))
    say("eight back-to-back calls on plans destroyed at once")
    outs = []
    for i in range(8):
        O = torch.empty((1, L, H, d), dtype=torch.float32, device="cuda")
        LSE = torch.empty((1, H, L), dtype=torch.float32, device="cuda")
        call(shapes[i % 4], O, LSE)
        outs.append((O, LSE))
    torch.cuda.synchronize()
    for i, (O, LSE) in enumerate(outs):
        assert torch.equal(O.cpu(), refs[i % 4][0]) and torch.equal(LSE.cpu(), refs[i % 4][1]), i
