"""Shared helpers of the GPU parity tests (no test functions here)."""
import sys

import numpy as np
import pytest
import torch

import paper_2604_20819_amd as cq
from paper_2604_20819_amd import synth


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")


def say(*a):
    """Name the case before GPU work starts (flushed, so a crash still shows it)."""
    print("[case]", *a, file=sys.stderr, flush=True)


def run_forward(Q, K, V, causal, depth=-1, budget=0, n_slots=2, host=False, scale=0.0,
                tasks_per_slot=0, levels=None, read_in_place=None):
    """Run cqsa_forward; Q, K, V are CPU tensors.  host=True keeps inputs and
    outputs in pinned host memory (streamed path).  Returns CPU (O, LSE, plan)."""
    B, L, H, d = Q.shape
    dt = {torch.float32: "f32", torch.float16: "f16", torch.bfloat16: "bf16"}[Q.dtype]
    opts = cq.make_opts(B=B, dtype=dt, depth=depth, n_slots=n_slots,
                        inputs_on_device=not host, acc_on_device=not host,
                        tasks_per_slot=tasks_per_slot, levels=levels,
                        read_in_place=read_in_place)
    plan = cq.cqsa_plan(L, H, d, causal, budget, opts)
    if host:
        q, k, v = (x.pin_memory() for x in (Q, K, V))
        O = torch.empty((B, L, H, d), dtype=torch.float32, pin_memory=True)
        LSE = torch.empty((B, H, L), dtype=torch.float32, pin_memory=True)
    else:
        q, k, v = (x.cuda() for x in (Q, K, V))
        O = torch.empty((B, L, H, d), dtype=torch.float32, device="cuda")
        LSE = torch.empty((B, H, L), dtype=torch.float32, device="cuda")
    cq.cqsa_forward(plan, q, k, v, O, LSE, scale)
    torch.cuda.synchronize()
    return O.cpu(), LSE.cpu(), plan


def reused_tokens(plan, reuse=True):
    """Tokens each staged task shares with the task staged just before it
    (interval intersection of the two tasks' global runs), summed over the
    plan; these are copied on the device instead of over the host link."""
    if not reuse:
        return 0
    total, prev = 0, None
    for t in range(plan.num_tasks):
        tk = plan.task(t)
        if tk["L_local"] == 0:
            continue
        runs = [(g, g + n) for g, n, _ in tk["runs"]]
        if prev is not None:
            total += sum(max(0, min(b1, b2) - max(a1, a2)) for a1, b1 in prev for a2, b2 in runs)
        prev = runs
    return total


def rel_l2(x, ref):
    x = np.asarray(x, dtype=np.float64); ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm((x - ref).ravel()) / np.linalg.norm(ref.ravel()))
