"""GPU tests of the kernels that read the caller's tensors in place.

With read_in_place the inner kernels address every task's runs inside the
caller's [B, L, H, d] tensors (a per-block row table for tiles inside one
run, per-lane rows for tiles that cross a run boundary) instead of first
gathering them into contiguous staging buffers (App. A.3 describes the
gather).  The arithmetic, the tile order and the values loaded are the same
either way, so results must be bit-identical to the staged path; parity
with the oracle follows from the staged path's own tests, and is also
checked here on the cases with the most run boundaries per tile.
"""
import numpy as np
import pytest
import torch

import paper_2604_20819_amd as cq
from paper_2604_20819_amd import synth
from tests.gpu_util import need_gpu, run_forward, say
from tests.test_gpu_backward import run_fwd_bwd
from tests.test_gpu_forward import _check_vs_oracle

pytestmark = pytest.mark.gpu

# (dtype, B, L, H, d, causal, depth, levels): short tasks and deep plans put
# run boundaries inside most tiles (depth 3 on 1500 tokens: ~4-token chunks)
FWD_CASES = [
    ("bf16", 1, 1, 2, 64, False, 1, None),
    ("bf16", 1, 100, 2, 64, True, 1, None),
    ("bf16", 2, 1000, 3, 128, True, 2, None),
    ("f16", 1, 2049, 2, 128, False, 2, None),
    ("bf16", 1, 1500, 2, 64, True, 3, None),
    ("f16", 2, 777, 2, 96, False, 2, None),
    ("bf16", 1, 3001, 2, 128, True, 2, [(13, (0, 1, 3, 9)), (7, (0, 1, 3))]),
    ("bf16", 1, 5000, 4, 256, False, 1, None),
    ("f32", 1, 1000, 2, 64, True, 2, None),
    ("f32", 2, 300, 1, 128, False, 1, None),
]


def _ids(cases):
    return ["-".join(str(x) for x in c[:7]) + ("-levels" if c[7] else "") for c in cases]


@pytest.mark.parametrize("dt,B,L,H,d,causal,depth,levels", FWD_CASES, ids=_ids(FWD_CASES))
def test_forward_in_place_equals_staged(dt, B, L, H, d, causal, depth, levels):
    need_gpu()
    Q, K, V = synth.make_inputs(71 + L, B, L, H, d, dt)
    say(f"in place forward {dt} B={B} L={L} H={H} d={d} causal={causal} depth={depth}")
    cq.cqsa_set_timing(True)
    try:
        O1, L1, p1 = run_forward(Q, K, V, causal, depth=depth, levels=levels, read_in_place=True)
        st = cq.cqsa_last_stats()
        O0, L0, p0 = run_forward(Q, K, V, causal, depth=depth, levels=levels, read_in_place=False)
        st0 = cq.cqsa_last_stats()
    finally:
        cq.cqsa_set_timing(False)
    assert p1.reads_in_place == 1 and p0.reads_in_place == 0
    assert st["d2d_bytes"] == 0 and st0["d2d_bytes"] > 0
    assert st["workspace_bytes"] < st0["workspace_bytes"]
    assert torch.equal(O1, O0) and torch.equal(L1, L0)
    assert np.isfinite(O1.numpy()).all()


@pytest.mark.parametrize("dt,causal", [("bf16", True), ("f16", False)])
def test_forward_in_place_vs_oracle_many_boundaries(dt, causal):
    need_gpu()
    B, L, H, d = 1, 1500, 2, 64
    Q, K, V = synth.make_inputs(83, B, L, H, d, dt)
    say(f"in place forward vs oracle {dt} causal={causal} depth 3")
    O, LSE, _ = run_forward(Q, K, V, causal, depth=3, read_in_place=True)
    _check_vs_oracle(O, LSE, Q, K, V, causal, dt)


BWD_CASES = [
    ("bf16", 1, 100, 2, 64, True, 1),
    ("bf16", 2, 1000, 2, 128, True, 2),
    ("f16", 1, 2049, 2, 128, False, 2),
    ("bf16", 1, 1500, 2, 64, False, 3),
    ("f16", 1, 900, 2, 96, True, 2),
    ("bf16", 1, 3000, 2, 256, True, 1),
]


@pytest.mark.parametrize("dt,B,L,H,d,causal,depth", BWD_CASES,
                         ids=["-".join(str(x) for x in c) for c in BWD_CASES])
def test_backward_in_place_equals_staged(dt, B, L, H, d, causal, depth):
    need_gpu()
    Q, K, V, dO = synth.make_inputs(91 + L, B, L, H, d, dt, with_dO=True)
    say(f"in place backward {dt} B={B} L={L} H={H} d={d} causal={causal} depth={depth}")
    cq.cqsa_set_timing(True)
    try:
        got = run_fwd_bwd(Q, K, V, dO, causal, depth=depth, read_in_place=True)
        st = cq.cqsa_last_stats()
        ref = run_fwd_bwd(Q, K, V, dO, causal, depth=depth, read_in_place=False)
        st0 = cq.cqsa_last_stats()
    finally:
        cq.cqsa_set_timing(False)
    assert got[-1].reads_in_place == 1 and ref[-1].reads_in_place == 0
    assert st["d2d_bytes"] == 0 and st0["d2d_bytes"] > 0
    # in place, the task-local gradients of a launch's tasks are what the
    # workspace holds (none with one task per launch)
    gs = got[-1].bwd_tasks_per_launch
    assert st["resident_tasks"] == (gs if gs > 1 else 0) and st0["resident_tasks"] > 0
    for name, g, r in zip(("O", "LSE", "dQ", "dK", "dV"), got[:5], ref[:5]):
        assert torch.equal(g, r), name
    assert all(np.isfinite(g.numpy()).all() for g in got[2:5])
