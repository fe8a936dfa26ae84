"""GPU tests of the 16-bit output option (out16).

With out16 the forward computes the same fp32 result as with an fp32 O and
rounds it once, to nearest even, into an O of the input dtype.  torch's
float32 -> bfloat16 / float16 conversions round the same way, so the 16-bit
O must equal the fp32 call's O converted by torch bit for bit, and LSE must
be identical.  Against the float64 oracle the 16-bit O carries the fp32
result's error (max-abs bound 1e-2) plus one rounding to the output dtype
(half an ulp: at most 2^-8 |O| for bf16, 2^-11 |O| for fp16), elementwise.
"""
import numpy as np
import pytest
import torch

import paper_2604_20819_amd as cq
from oracle import dense
from paper_2604_20819_amd import synth
from tests.gpu_util import need_gpu, say

pytestmark = pytest.mark.gpu

# (dtype, B, L, H, d, causal, depth, read_in_place, host-resident inputs)
CASES = [
    ("bf16", 1, 1, 2, 64, False, 0, None, False),
    ("bf16", 2, 1000, 3, 128, True, 0, None, False),
    ("f16", 1, 2049, 2, 128, False, 1, None, False),
    ("bf16", 1, 3000, 4, 96, True, 2, True, False),
    ("f16", 2, 777, 2, 256, False, 2, False, False),
    ("bf16", 1, 1500, 2, 64, True, 1, False, True),
]


@pytest.mark.parametrize("dt,B,L,H,d,causal,depth,rip,host_in", CASES,
                         ids=["-".join(map(str, c)) for c in CASES])
def test_out16_equals_rounded_fp32(dt, B, L, H, d, causal, depth, rip, host_in):
    need_gpu()
    say(f"out16 {dt} B={B} L={L} H={H} d={d} causal={causal} depth={depth} "
        f"read_in_place={rip} host_inputs={host_in}")
    Q, K, V = synth.make_inputs(4242 + L, B, L, H, d, dt)
    tdt = Q.dtype
    if host_in:
        q, k, v = (x.pin_memory() for x in (Q, K, V))
    else:
        q, k, v = (x.cuda() for x in (Q, K, V))
    res = {}
    for out16 in (False, True):
        opts = cq.make_opts(B=B, dtype=dt, depth=depth, inputs_on_device=not host_in,
                            acc_on_device=True, read_in_place=rip, out16=out16)
        plan = cq.cqsa_plan(L, H, d, causal, 0, opts)
        O = torch.full((B, L, H, d), float("nan"), dtype=tdt if out16 else torch.float32,
                       device="cuda")
        LSE = torch.full((B, H, L), float("nan"), dtype=torch.float32, device="cuda")
        cq.cqsa_forward(plan, q, k, v, O, LSE)
        torch.cuda.synchronize()
        res[out16] = (O.cpu(), LSE.cpu())
    (o32, l32), (o16, l16) = res[False], res[True]
    assert o16.dtype == tdt
    assert torch.equal(o16, o32.to(tdt))
    assert torch.equal(l16, l32)
    Of, Lf = dense.attention_forward(synth.as_f64(Q), synth.as_f64(K), synth.as_f64(V), causal)
    half_ulp = {"bf16": 2.0 ** -8, "f16": 2.0 ** -11}[dt]
    err = np.abs(o16.double().numpy() - Of)
    say(f"  max |O16 - O64| = {err.max():.3e}, max |LSE - LSE64| = "
        f"{np.abs(l16.double().numpy() - Lf).max():.3e}")
    assert (err <= 1e-2 + half_ulp * np.abs(Of)).all()
    assert np.abs(l16.double().numpy() - Lf).max() <= 1e-4


def test_out16_back_to_back_calls_share_the_workspace():
    """Two out16 calls of different plans in a row, the second smaller: each
    call's fp32 result lives in the shared workspace, and the second must not
    see the first's."""
    need_gpu()
    outs = []
    for L in (4000, 1500):
        say(f"out16 back-to-back L={L}")
        Q, K, V = synth.make_inputs(77 + L, 1, L, 2, 128, "bf16")
        q, k, v = (x.cuda() for x in (Q, K, V))
        ref = []
        for out16 in (False, True):
            plan = cq.cqsa_plan(L, 2, 128, True, 0, cq.make_opts(dtype="bf16", depth=1, out16=out16))
            O = torch.empty((1, L, 2, 128), dtype=torch.bfloat16 if out16 else torch.float32,
                            device="cuda")
            LSE = torch.empty((1, 2, L), dtype=torch.float32, device="cuda")
            cq.cqsa_forward(plan, q, k, v, O, LSE)
            ref.append(O)
        torch.cuda.synchronize()
        outs.append(torch.equal(ref[1].cpu(), ref[0].cpu().to(torch.bfloat16)))
    assert outs == [True, True]
