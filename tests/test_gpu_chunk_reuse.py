"""GPU tests of chunk reuse when host-resident inputs are staged.

Consecutive tasks in quorum order share chunks (at depth 1 with
I = (0, 1, 3), task q + 1 holds chunk q + 1 of task q).  When a task's runs
are staged from host memory, the tokens the previously staged task also
holds are copied device to device from that task's staged rows, and only
the rest crosses the host link.  The staged rows, and so every result, are
the same as a full gather: outputs must be bit-identical to staging the same
plan from device-resident inputs, and the host-link bytes must equal the
task tokens minus the shared ones (computed here from the plan's runs).
"""
import numpy as np
import pytest
import torch

import paper_2604_20819_amd as cq
from paper_2604_20819_amd import synth
from tests.gpu_util import need_gpu, rel_l2, reused_tokens, run_forward, say
from tests.test_gpu_forward import _check_vs_oracle

pytestmark = pytest.mark.gpu


def _forward(Q, K, V, causal, depth, tps, n_slots, host_inputs):
    """Device accumulator; inputs on the host (pinned) or staged from device."""
    B, L, H, d = Q.shape
    dt = {torch.float16: "f16", torch.bfloat16: "bf16"}[Q.dtype]
    plan = cq.cqsa_plan(L, H, d, causal, 0,
                        cq.make_opts(B=B, dtype=dt, depth=depth, n_slots=n_slots,
                                     inputs_on_device=not host_inputs, tasks_per_slot=tps,
                                     read_in_place=False))
    if host_inputs:
        q, k, v = (x.pin_memory() for x in (Q, K, V))
    else:
        q, k, v = (x.cuda() for x in (Q, K, V))
    O = torch.empty((B, L, H, d), dtype=torch.float32, device="cuda")
    LSE = torch.empty((B, H, L), dtype=torch.float32, device="cuda")
    cq.cqsa_set_timing(True)
    try:
        cq.cqsa_forward(plan, q, k, v, O, LSE)
        torch.cuda.synchronize()
        st = cq.cqsa_last_stats()
    finally:
        cq.cqsa_set_timing(False)
    return O.cpu(), LSE.cpu(), plan, st


# (dtype, B, L, H, d, causal, depth, tasks per launch, slots): with one slot
# and one task per launch consecutive tasks share a sub-slot, so nothing is
# reused; every other grouping reuses within and across launch groups
CASES = [
    ("bf16", 1, 3001, 2, 64, False, 1, 1, 2),
    ("bf16", 2, 3001, 2, 128, True, 2, 1, 2),
    ("f16", 1, 2049, 3, 64, True, 2, 5, 2),
    ("bf16", 1, 5000, 2, 128, False, 1, 3, 1),
    ("bf16", 1, 1000, 2, 64, True, 2, 1, 1),
    ("f16", 2, 1500, 2, 96, False, 3, 8, 3),
]


@pytest.mark.parametrize("dt,B,L,H,d,causal,depth,tps,n_slots", CASES,
                         ids=["-".join(str(x) for x in c) for c in CASES])
def test_reuse_matches_device_staging(dt, B, L, H, d, causal, depth, tps, n_slots):
    need_gpu()
    Q, K, V = synth.make_inputs(101 + L, B, L, H, d, dt)
    say(f"chunk reuse {dt} B={B} L={L} H={H} d={d} causal={causal} depth={depth} "
        f"tps={tps} slots={n_slots}")
    Oh, Lh, plan, st = _forward(Q, K, V, causal, depth, tps, n_slots, True)
    Od, Ld, _, std = _forward(Q, K, V, causal, depth, tps, n_slots, False)
    assert torch.equal(Oh, Od) and torch.equal(Lh, Ld)
    row = H * d * 2
    tokens = sum(plan.task(t)["L_local"] for t in range(plan.num_tasks))
    reuse = not (n_slots == 1 and plan.tasks_per_slot == 1)
    shared = reused_tokens(plan, reuse)
    say(f"  task tokens {tokens}, reused {shared}")
    assert st["h2d_bytes"] == 3 * B * (tokens - shared) * row
    assert st["d2d_bytes"] == 3 * B * shared * row
    assert std["d2d_bytes"] == 3 * B * tokens * row and std["h2d_bytes"] == 0
    if reuse:
        assert shared > 0
    _check_vs_oracle(Oh, Lh, Q, K, V, causal, dt)


def test_streamed_host_accumulator_reuses_chunks():
    """The streamed path (host inputs and outputs) stages with reuse and
    matches the device-resident call."""
    need_gpu()
    Q, K, V = synth.make_inputs(113, 2, 4001, 2, 64, "bf16")
    say("chunk reuse, host inputs and outputs, depth 2")
    cq.cqsa_set_timing(True)
    try:
        O, LSE, plan = run_forward(Q, K, V, True, depth=2, host=True)
        st = cq.cqsa_last_stats()
    finally:
        cq.cqsa_set_timing(False)
    tokens = sum(plan.task(t)["L_local"] for t in range(plan.num_tasks))
    shared = reused_tokens(plan)
    assert shared > 0.25 * tokens
    assert st["h2d_bytes"] == 3 * 2 * (tokens - shared) * 2 * 64 * 2
    Od, Ld, _ = run_forward(Q, K, V, True, depth=2)
    assert rel_l2(O.numpy(), Od.numpy()) <= 1e-6
    assert np.abs(LSE.numpy() - Ld.numpy()).max() <= 1e-5
