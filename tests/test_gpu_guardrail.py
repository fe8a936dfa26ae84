"""GPU tests of the OOM guardrail (Section 3.4, "OOM guardrails").

Allocation failures are forced from the host: a caller allocator (the
cqsa_set_allocator hook) refuses requests above a limit and returns NULL, so
the library sees CQSA_ERR_DEVICE_OOM before it enqueues any work.  With an
automatic depth the call must then succeed with fewer resident task working
sets or a deeper plan, and match both the float64 oracle and the
unconstrained result; a forced depth must report the failure.
"""
import numpy as np
import pytest
import torch

import paper_2604_20819_amd as cq
from paper_2604_20819_amd import synth
from tests.gpu_util import need_gpu, rel_l2, say
from tests.test_gpu_backward import _check_grads, oracle_grads
from tests.test_gpu_forward import _check_vs_oracle

pytestmark = pytest.mark.gpu


class LimitedAllocator:
    """Serves torch device memory up to `limit` bytes per request."""

    def __init__(self, limit):
        self.limit, self.held, self.refused, self.served = limit, {}, 0, []

    def alloc(self, n):
        if n > self.limit:
            self.refused += 1
            return 0
        t = torch.empty((n,), dtype=torch.uint8, device="cuda")
        self.held[t.data_ptr()] = t
        self.served.append(n)
        return t.data_ptr()

    def release(self, ptr):
        self.held.pop(ptr)

    def __enter__(self):
        cq.cqsa_set_allocator(self.alloc, self.release)
        return self

    def __exit__(self, *exc):
        cq.cqsa_set_allocator(None, None)


def _forward(plan, q, k, v):
    B, L, H, d = q.shape
    O = torch.empty((B, L, H, d), dtype=torch.float32, device="cuda")
    LSE = torch.empty((B, H, L), dtype=torch.float32, device="cuda")
    cq.cqsa_forward(plan, q, k, v, O, LSE)
    torch.cuda.synchronize()
    return O.cpu(), LSE.cpu()


def test_forward_guardrail_lowers_residency_then_deepens():
    need_gpu()
    L, H, d = 3000, 2, 128
    Q, K, V = synth.make_inputs(41, 1, L, H, d, "bf16")
    q, k, v = (x.cuda() for x in (Q, K, V))
    say("guardrail forward: unconstrained run")
    cq.cqsa_set_timing(True)
    try:
        plan = cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(dtype="bf16"))
        O0, L0 = _forward(plan, q, k, v)
        st0 = cq.cqsa_last_stats()
        assert st0["guard_steps"] == 0 and plan.depth == 1
        full = st0["workspace_bytes"]
        limit = full // 3
        say(f"guardrail forward: workspace {full} B, limit {limit} B")
        with LimitedAllocator(limit) as a:
            O1, L1 = _forward(plan, q, k, v)
            st1 = cq.cqsa_last_stats()
            say(f"  fallbacks {st1['guard_steps']}, depth {st1['depth']}, "
                f"resident {st1['resident_tasks']}, workspace {st1['workspace_bytes']} B")
            assert a.refused >= 1 and st1["guard_steps"] >= 1
            assert st1["workspace_bytes"] <= limit and a.served == [st1["workspace_bytes"]]
            assert st1["resident_tasks"] < st0["resident_tasks"] or st1["depth"] > 1
            # later calls start from the configuration that succeeded
            refused = a.refused
            O2, L2 = _forward(plan, q, k, v)
            st2 = cq.cqsa_last_stats()
            assert a.refused == refused and st2["guard_steps"] == 0
            assert st2["depth"] == st1["depth"] and st2["workspace_bytes"] == st1["workspace_bytes"]
            assert not a.held
    finally:
        cq.cqsa_set_timing(False)
    for O, LSE in ((O1, L1), (O2, L2)):
        assert rel_l2(O.numpy(), O0.numpy()) <= 2e-5
        assert np.abs(LSE.numpy() - L0.numpy()).max() <= 1e-5
        _check_vs_oracle(O, LSE, Q, K, V, False, "bf16")


def test_forward_guardrail_reaches_a_deeper_level():
    """A limit below every depth-1 configuration forces depth 2."""
    need_gpu()
    L, H, d = 3000, 2, 128
    Q, K, V = synth.make_inputs(42, 1, L, H, d, "bf16")
    q, k, v = (x.cuda() for x in (Q, K, V))
    ref = cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(dtype="bf16", depth=0))
    O0, L0 = _forward(ref, q, k, v)
    one = cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(dtype="bf16", depth=1, n_slots=1,
                                                        tasks_per_slot=1))
    cq.cqsa_set_timing(True)
    try:
        _forward(one, q, k, v)
        smallest_depth1 = cq.cqsa_last_stats()["workspace_bytes"]
        plan = cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(dtype="bf16"))
        with LimitedAllocator(smallest_depth1 - 1):
            say("guardrail forward: limit below every depth-1 configuration")
            O, LSE = _forward(plan, q, k, v)
            st = cq.cqsa_last_stats()
    finally:
        cq.cqsa_set_timing(False)
    say(f"  fallbacks {st['guard_steps']}, depth {st['depth']}")
    assert st["depth"] == 2 and st["workspace_bytes"] < smallest_depth1
    assert rel_l2(O.numpy(), O0.numpy()) <= 2e-5
    assert np.abs(LSE.numpy() - L0.numpy()).max() <= 1e-5
    _check_vs_oracle(O, LSE, Q, K, V, False, "bf16")


def test_forced_depth_reports_the_failure_and_exhaustion_is_reported():
    need_gpu()
    L, H, d = 2000, 2, 128
    Q, K, V = synth.make_inputs(43, 1, L, H, d, "bf16")
    q, k, v = (x.cuda() for x in (Q, K, V))
    forced = cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(dtype="bf16", depth=1))
    auto = cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(dtype="bf16", max_depth=2))
    with LimitedAllocator(1024) as a:
        say("guardrail: forced depth with a 1 KB limit")
        with pytest.raises(cq.CqsaError) as e:
            _forward(forced, q, k, v)
        assert e.value.status == -4 and a.refused == 1
        say("guardrail: automatic depth with a 1 KB limit (exhausted at max_depth 2)")
        with pytest.raises(cq.CqsaError) as e:
            _forward(auto, q, k, v)
        assert e.value.status == -4 and "guardrail" in str(e.value) and a.refused > 2
        assert not a.held
    # the device is still usable and the plan still works without the limit
    O, _ = _forward(auto, q, k, v)
    assert np.isfinite(O.numpy()).all()


def test_backward_guardrail():
    """The backward's resident task working sets are its staging slots, so
    the plan gathers its inputs (read in place it holds none)."""
    need_gpu()
    L, H, d = 2500, 2, 128
    Q, K, V, dO = synth.make_inputs(44, 1, L, H, d, "bf16", with_dO=True)
    q, k, v, do = (x.cuda() for x in (Q, K, V, dO))
    plan = cq.cqsa_plan(L, H, d, True, 0, cq.make_opts(dtype="bf16", with_backward=True,
                                                       read_in_place=False))
    O = torch.empty((1, L, H, d), dtype=torch.float32, device="cuda")
    LSE = torch.empty((1, H, L), dtype=torch.float32, device="cuda")
    cq.cqsa_forward(plan, q, k, v, O, LSE)

    def grads():
        g = [torch.empty((1, L, H, d), dtype=torch.float32, device="cuda") for _ in range(3)]
        cq.cqsa_backward(plan, q, k, v, O, LSE, do, *g)
        torch.cuda.synchronize()
        return [x.cpu() for x in g]

    cq.cqsa_set_timing(True)
    try:
        ref = grads()
        full = cq.cqsa_last_stats()["workspace_bytes"]
        with LimitedAllocator(full - 1) as a:
            say(f"guardrail backward: workspace {full} B, limit {full - 1} B")
            got = grads()
            st = cq.cqsa_last_stats()
            assert a.refused >= 1 and st["guard_steps"] >= 1 and st["workspace_bytes"] < full
    finally:
        cq.cqsa_set_timing(False)
    say(f"  fallbacks {st['guard_steps']}, depth {st['depth']}, resident {st['resident_tasks']}")
    for g, r in zip(got, ref):
        assert rel_l2(g.numpy(), r.numpy()) <= 1e-3
    _check_grads(got, oracle_grads(Q, K, V, dO, True), "bf16")


def test_batched_backward_guardrail():
    """Read in place, the backward's resident task working sets are the
    task-local gradients of one launch group: a refused workspace halves the
    tasks per launch (7 -> 3), and since every grouping adds the same values in
    the same order the gradients keep their bits."""
    need_gpu()
    L, H, d = 2500, 2, 128
    Q, K, V, dO = synth.make_inputs(45, 1, L, H, d, "bf16", with_dO=True)
    q, k, v, do = (x.cuda() for x in (Q, K, V, dO))
    plan = cq.cqsa_plan(L, H, d, True, 0, cq.make_opts(dtype="bf16", with_backward=True))
    assert plan.reads_in_place == 1 and plan.bwd_tasks_per_launch == 7
    O = torch.empty((1, L, H, d), dtype=torch.float32, device="cuda")
    LSE = torch.empty((1, H, L), dtype=torch.float32, device="cuda")
    cq.cqsa_forward(plan, q, k, v, O, LSE)

    def grads():
        g = [torch.empty((1, L, H, d), dtype=torch.float32, device="cuda") for _ in range(3)]
        cq.cqsa_backward(plan, q, k, v, O, LSE, do, *g)
        torch.cuda.synchronize()
        return [x.cpu() for x in g]

    cq.cqsa_set_timing(True)
    try:
        ref = grads()
        st0 = cq.cqsa_last_stats()
        full = st0["workspace_bytes"]
        with LimitedAllocator(full - 1) as a:
            say(f"guardrail batched backward: workspace {full} B, limit {full - 1} B")
            got = grads()
            st = cq.cqsa_last_stats()
            assert a.refused >= 1 and st["guard_steps"] == 1 and st["workspace_bytes"] < full
    finally:
        cq.cqsa_set_timing(False)
    say(f"  fallbacks {st['guard_steps']}, depth {st['depth']}, resident {st0['resident_tasks']}"
        f" -> {st['resident_tasks']}")
    assert st0["resident_tasks"] == 7 and st["resident_tasks"] == 3 and st["depth"] == 1
    for g, r in zip(got, ref):
        assert torch.equal(g, r)
    _check_grads(got, oracle_grads(Q, K, V, dO, True), "bf16")


def test_host_resident_backward_guardrail():
    """With every tensor in host memory the backward's staging slots hold the
    task's inputs and its own gradients; a workspace refusal drops to one
    slot (or a deeper plan), and the gradients still match float64."""
    need_gpu()
    L, H, d = 2500, 2, 64
    Q, K, V, dO = synth.make_inputs(45, 1, L, H, d, "bf16", with_dO=True)
    q, k, v, do = (x.pin_memory() for x in (Q, K, V, dO))
    plan = cq.cqsa_plan(L, H, d, True, 0, cq.make_opts(dtype="bf16", with_backward=True,
                                                       inputs_on_device=False,
                                                       acc_on_device=False))
    O = torch.empty((1, L, H, d), dtype=torch.float32, pin_memory=True)
    LSE = torch.empty((1, H, L), dtype=torch.float32, pin_memory=True)
    cq.cqsa_forward(plan, q, k, v, O, LSE)

    def grads():
        g = [torch.empty((1, L, H, d), dtype=torch.float32, pin_memory=True) for _ in range(3)]
        cq.cqsa_backward(plan, q, k, v, O, LSE, do, *g)
        return g

    cq.cqsa_set_timing(True)
    try:
        ref = grads()
        full = cq.cqsa_last_stats()["workspace_bytes"]
        with LimitedAllocator(full - 1) as a:
            say(f"guardrail host backward: workspace {full} B, limit {full - 1} B")
            got = grads()
            st = cq.cqsa_last_stats()
            assert a.refused >= 1 and st["guard_steps"] >= 1 and st["workspace_bytes"] < full
            assert not a.held
    finally:
        cq.cqsa_set_timing(False)
    say(f"  fallbacks {st['guard_steps']}, depth {st['depth']}, resident {st['resident_tasks']}")
    for g, r in zip(got, ref):
        assert rel_l2(g.numpy(), r.numpy()) <= 1e-3
    _check_grads(got, oracle_grads(Q, K, V, dO, True), "bf16")
