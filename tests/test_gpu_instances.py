"""GPU tests: every compiled instance of the attention kernels at every head
dim gives the same bits as its siblings.

Each kernel is built in instances that a call picks by its plan and flags:
the backward kernels with their task-local epilogue (several tasks per
launch) or with the read-modify-write into the global gradients (one task
per launch), each with and without tile counting; the forward with and
without counting.  Their arithmetic is the same, so all of them must give the
same bits; a fault in one instance's compiled code (as a misplaced register
spill once caused in one of them) shows as a difference.  One result per
head dim is also held to float64.
"""
import numpy as np
import pytest
import torch

import paper_2604_20819_amd as cq
from paper_2604_20819_amd import synth
from tests.gpu_util import need_gpu, rel_l2, say
from tests.test_gpu_backward import REL, oracle_grads

pytestmark = pytest.mark.gpu

DIMS = [32, 64, 96, 128, 160, 192, 224, 256]


def call(plan, q, k, v, do, B, L, H, d, counting):
    O = torch.full((B, L, H, d), float("nan"), dtype=torch.float32, device="cuda")
    LSE = torch.full((B, H, L), float("nan"), dtype=torch.float32, device="cuda")
    g = [torch.full((B, L, H, d), float("nan"), dtype=torch.float32, device="cuda") for _ in range(3)]
    cq.cqsa_set_tile_counting(counting)
    try:
        cq.cqsa_forward(plan, q, k, v, O, LSE)
        cq.cqsa_backward(plan, q, k, v, O, LSE, do, *g)
        torch.cuda.synchronize()
    finally:
        cq.cqsa_set_tile_counting(False)
    return [x.cpu() for x in [O, LSE] + g]


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("d", DIMS)
def test_every_instance_gives_the_same_bits(d, dt):
    need_gpu()
    B, L, H, causal = 1, 1100, 2, True
    say(f"kernel instances {dt} d={d} B={B} L={L} H={H} causal")
    Q, K, V, dO = synth.make_inputs(7300 + d + (dt == "f16"), B, L, H, d, dt, with_dO=True)
    q, k, v, do = (x.cuda() for x in (Q, K, V, dO))
    res = {}
    for tpl in (0, 1):
        plan = cq.cqsa_plan(L, H, d, causal, 0,
                            cq.make_opts(B=B, dtype=dt, depth=1, with_backward=True, bwd_tasks_per_launch=tpl))
        for counting in (False, True):
            res[(tpl, counting)] = call(plan, q, k, v, do, B, L, H, d, counting)
    ref = res[(0, False)]
    names = ("O", "LSE", "dQ", "dK", "dV")
    for key, out in res.items():
        for name, a, b in zip(names, out, ref):
            assert torch.isfinite(a).all(), (key, name)
            assert torch.equal(a, b), (key, name)
    want = oracle_grads(Q, K, V, dO, causal)
    for name, g, w in zip(("dQ", "dK", "dV"), ref[2:], want):
        r = rel_l2(g.numpy(), w)
        say(f"  {name} vs float64: {r:.3e}")
        assert r <= 2e-2 and r <= REL[dt], name
