"""C-ABI tests that need no GPU: the library loads and exports every symbol
include/cqsa.h declares; planning through the ABI is bit-exact against the
independent oracle planner; argument validation; the footprint model picks
the depths the workload definitions call for."""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

import paper_2604_20819_amd as cq
from oracle import planner as oplan
from tests.conftest import ROOT


def _declared_symbols():
    text = open(os.path.join(ROOT, "include", "cqsa.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cqsa_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = cq.lib()
    syms = _declared_symbols()
    assert "cqsa_forward" in syms and "cqsa_backward" in syms and "cqsa_plan" in syms
    for s in syms:
        assert hasattr(lib, s), s
        assert s in cq._SIGS, s


@pytest.mark.parametrize("N,itr,c", [(7, 1, 7), (49, 2, 7), (100, 1, 7), (100, 2, 7),
                                      (343, 3, 7), (1000, 2, 7), (65536, 1, 7), (5000, 2, 7),
                                      (90, 2, 13), (13, 1, 13), (30, 1, 3), (10, 0, 7)])
def test_planner_matches_oracle(N, itr, c):
    I = oplan.PAPER_INTEREST_SETS[c] if c in oplan.PAPER_INTEREST_SETS else (0, 1)
    p = cq.cqsa_plan(N, 1, 64, False, 0, cq.make_opts(c=c, interest=I, depth=itr))
    ref = oplan.build_tasks(N, c, itr, I)
    assert p.depth == itr and p.num_tasks == len(ref) == c ** itr
    for t, rt in enumerate(ref):
        got = p.task(t)
        assert got["quorum"] == tuple(rt["quorum"])
        assert got["L_local"] == len(rt["tokens"])
        assert got["runs"] == oplan.runs(rt)
        bor, band = oplan.block_summaries(rt["bits"])
        assert got["block_or"] == bor.tolist() and got["block_and"] == band.tolist()


@pytest.mark.parametrize("N,levels,depth", [
    (500, [(7, (0, 1, 3)), (13, (0, 1, 3, 9))], 2),
    (500, [(13, (0, 1, 3, 9)), (7, (0, 1, 3))], 2),
    (3000, [(21, (0, 1, 4, 14, 16)), (3, (0, 1))], 2),
    (700, [(3, (0, 1)), (7, (0, 1, 3))], 3),        # the last set repeats below
    (65536, [(13, (0, 1, 3, 9))], 1),
    (90, [(7, (0, 1, 3)), (13, (0, 1, 3, 9)), (3, (0, 1))], 3)])
def test_planner_matches_oracle_with_level_sets(N, levels, depth):
    """Section 3.3: a different valid interest set per depth.  Tasks, runs,
    bits and block summaries equal the oracle planner's."""
    p = cq.cqsa_plan(N, 1, 64, False, 0, cq.make_opts(depth=depth, levels=levels))
    full = (levels + [levels[-1]] * depth)[:depth]
    ref = oplan.build_tasks_levels(N, full)
    assert p.depth == depth and p.num_tasks == len(ref)
    for t, rt in enumerate(ref):
        got = p.task(t)
        assert got["quorum"] == tuple(rt["quorum"])
        assert got["runs"] == oplan.runs(rt)
        bor, band = oplan.block_summaries(rt["bits"])
        assert got["block_or"] == bor.tolist() and got["block_and"] == band.tolist()


@pytest.mark.parametrize("levels,depth,status,msg", [
    ([(7, (0, 1, 3)), (13, (0, 1, 3, 4))], 2, -1, "level set 1"),
    ([(7, (0, 1, 3)), (12, (0, 1, 3, 9))], 2, -1, "c must equal"),
    ([(21, (0, 1, 4, 14, 16))], 9, -2, "group bits exceed 32"),
    ([(13, (0, 1, 3, 9)), (7, (0, 1, 3))], 7, -2, "2^20 tasks")])
def test_level_set_errors(levels, depth, status, msg):
    with pytest.raises(cq.CqsaError) as e:
        cq.cqsa_plan(1000, 1, 64, False, 0, cq.make_opts(depth=depth, levels=levels))
    assert e.value.status == status and msg in str(e.value)
    o = cq.make_opts()
    o.n_level_sets = 5
    with pytest.raises(cq.CqsaError) as e:
        cq.cqsa_plan(1000, 1, 64, False, 0, o)
    assert e.value.status == -1


@pytest.mark.parametrize("d", [32, 64, 96, 128, 160, 192, 224, 256])
def test_forward_head_dims_accepted(d):
    p = cq.cqsa_plan(1000, 2, d, False, 0, cq.make_opts(depth=1))
    assert p.depth == 1 and p.num_tasks == 7


@pytest.mark.parametrize("d,backward", [(48, False), (288, False), (0, False), (80, True),
                                        (320, True)])
def test_head_dims_refused(d, backward):
    """Forward and backward: multiples of 32 up to 256 (Sec. 5)."""
    with pytest.raises(cq.CqsaError) as e:
        cq.cqsa_plan(1000, 2, d, False, 0, cq.make_opts(with_backward=backward))
    assert e.value.status in (-1, -2)


def test_automatic_accumulator_residency():
    """App. A.3: residency moves the accumulator off the device when no depth
    fits the budget with it there.  The 1M-token bf16 call with host inputs
    and a 4 GB budget cannot hold its 4.3 GB fp32 output on the device."""
    GB = 10 ** 9
    p = cq.cqsa_plan(32768, 16, 128, False, 0, cq.make_opts(acc_on_device=None))
    assert p.acc_on_device == 1 and p.depth == 1
    p = cq.cqsa_plan(1 << 20, 8, 128, False, 4 * GB,
                     cq.make_opts(acc_on_device=None, inputs_on_device=False))
    assert p.acc_on_device == 0 and p.depth == 2 and p.modelled_device_bytes <= 4 * GB
    # a forced depth keeps the device when it fits there, else goes to the host
    p = cq.cqsa_plan(1 << 20, 8, 128, False, 4 * GB,
                     cq.make_opts(acc_on_device=None, inputs_on_device=False, depth=3))
    assert p.acc_on_device == 0 and p.depth == 3
    # with the backward: the gradients follow the accumulator (Table
    # "recovery": fwd+bwd with the accumulator on the host)
    p = cq.cqsa_plan(4096, 4, 128, False, 0, cq.make_opts(acc_on_device=None, with_backward=True))
    assert p.acc_on_device == 1
    p = cq.cqsa_plan(1 << 20, 8, 128, True, 8 * GB,
                     cq.make_opts(acc_on_device=None, inputs_on_device=False, with_backward=True))
    assert p.acc_on_device == 0 and p.modelled_device_bytes <= 8 * GB


def test_read_in_place_choice_and_errors():
    """The kernels read the caller's tensors in place when they are on the
    device and a batch element's [L, H, d] slice spans under 2^31 bytes (the
    reach of a buffer load's 32-bit offset); otherwise runs are gathered."""
    p = cq.cqsa_plan(32768, 16, 128, False, 0, cq.make_opts())
    assert p.reads_in_place == 1
    p = cq.cqsa_plan(32768, 16, 128, False, 0, cq.make_opts(read_in_place=False))
    assert p.reads_in_place == 0
    p = cq.cqsa_plan(32768, 16, 128, False, 0, cq.make_opts(inputs_on_device=False,
                                                            acc_on_device=False))
    assert p.reads_in_place == 0
    # 2^20 x 8 x 128 x 2 bytes = 2^31: one byte past the reach
    p = cq.cqsa_plan(1 << 20, 8, 128, False, 0, cq.make_opts(depth=2))
    assert p.reads_in_place == 0
    p = cq.cqsa_plan((1 << 20) - 1, 8, 128, False, 0, cq.make_opts(depth=2))
    assert p.reads_in_place == 1
    p = cq.cqsa_plan(1 << 19, 8, 128, False, 0, cq.make_opts(depth=2, dtype="f32"))
    assert p.reads_in_place == 0
    for kw, status in [(dict(read_in_place=True, inputs_on_device=False, acc_on_device=False), -2),
                       (dict(read_in_place=True, depth=2), -2)]:
        with pytest.raises(cq.CqsaError) as e:
            cq.cqsa_plan(1 << 20, 8, 128, False, 0, cq.make_opts(**kw))
        assert e.value.status == status and "read_in_place" in str(e.value)
    o = cq.make_opts()
    o.read_in_place = 2
    with pytest.raises(cq.CqsaError) as e:
        cq.cqsa_plan(4096, 4, 64, False, 0, o)
    assert e.value.status == -1
    # in place, one backward task per launch holds no staging slots: the
    # forward's sub-slots are the peak, and they shrink by the three staged
    # inputs
    kw = dict(B=2, with_backward=True, depth=1)
    a = cq.cqsa_plan(65536, 16, 128, True, 0, cq.make_opts(bwd_tasks_per_launch=1, **kw))
    b = cq.cqsa_plan(65536, 16, 128, True, 0, cq.make_opts(read_in_place=False, **kw))
    assert a.bwd_tasks_per_launch == 1 and b.bwd_tasks_per_launch == 1
    assert a.modelled_device_bytes < b.modelled_device_bytes


def test_struct_layouts_match_the_header(tmp_path):
    """The binding's ctypes mirrors have the sizes and field offsets of the C
    structs in include/cqsa.h (checked by compiling the header with gcc)."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    checks = {"cqsa_plan_opts": ["B", "interest", "tasks_per_slot", "n_level_sets", "level_sets",
                                 "out16", "bwd_tasks_per_launch"],
              "cqsa_interest_set": ["c", "l", "interest"],
              "cqsa_tensor": ["data", "B", "d"], "cqsa_task": ["quorum", "runs", "block_and"],
              "cqsa_run": ["global_start", "bits"],
              "cqsa_run_stats": ["num_tasks", "ms_wall", "tiles_mixed", "ms_inner_busy",
                                 "guard_steps", "resident_tasks"]}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "cqsa.h"', "int main(void) {"]
    for st, fields in checks.items():
        lines.append(f'  printf("{st} %zu\\n", sizeof({st}));')
        for f in fields:
            lines.append(f'  printf("{st}.{f} %zu\\n", offsetof({st}, {f}));')
    lines.append("  return 0;\n}")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    inc = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
    subprocess.run(["gcc", "-std=c11", "-I", inc, str(src), "-o", str(exe)], check=True)
    got = dict(l.split() for l in subprocess.run([str(exe)], check=True, capture_output=True,
                                                 text=True).stdout.splitlines())
    for st, fields in checks.items():
        cls = getattr(cq, st)
        assert int(got[st]) == ctypes.sizeof(cls), st
        for f in fields:
            assert int(got[f"{st}.{f}"]) == getattr(cls, f).offset, (st, f)


@pytest.mark.parametrize("N,itr", [(65536, 1), (65536, 2), (20000, 3)])
def test_census_matches_oracle(N, itr):
    p = cq.cqsa_plan(N, 1, 64, True, 0, cq.make_opts(depth=itr))
    f, c, m, _ = oplan.tile_census(oplan.build_tasks(N, 7, itr, (0, 1, 3)))
    assert p.tile_census() == (f, c, m)


@pytest.mark.parametrize("kw,budget,msg", [
    (dict(interest=(0, 1, 2)), 0, "difference set"),
    (dict(c=8), 0, "l(l-1)+1"),
    (dict(n_slots=0), 0, "n_slots"),
    (dict(depth=-2), 0, "depth"),
    (dict(min_depth=3, max_depth=2), 0, "min_depth"),
])
def test_plan_rejects_bad_options(kw, budget, msg):
    with pytest.raises(cq.CqsaError) as e:
        cq.cqsa_plan(1000, 2, 64, False, budget, cq.make_opts(**kw))
    assert e.value.status == -1 and msg in str(e.value)


def test_plan_rejects_bad_geometry():
    with pytest.raises(cq.CqsaError) as e:
        cq.cqsa_plan(0, 2, 64, False, 0)
    assert e.value.status == -1
    with pytest.raises(cq.CqsaError) as e:
        cq.cqsa_plan(100, 2, 80, False, 0)
    assert e.value.status == -2
    with pytest.raises(cq.CqsaError) as e:
        cq.cqsa_plan(100, 2, 64, False, 0, cq.make_opts(depth=9))
    assert e.value.status == -2


def test_budget_too_small():
    with pytest.raises(cq.CqsaError) as e:
        cq.cqsa_plan(1 << 20, 8, 128, False, 1 << 20, cq.make_opts(max_depth=3))
    assert e.value.status == -3


GB = 10 ** 9
# (L, H, d, causal, budget, opts, expected depth) for the five workloads; the
# 8 GB fp16 causal call needs depth 2 when every task's inputs are staged and
# fits at depth 1 when the kernels read the caller's tensors in place
WORKLOADS = [
    (1024, 1, 64, False, 0, dict(dtype="f32", depth=1), 1),
    (32768, 16, 128, False, 0, dict(dtype="bf16", depth=1), 1),
    (131072, 32, 128, True, 8 * GB, dict(dtype="f16", read_in_place=False), 2),
    (131072, 32, 128, True, 8 * GB, dict(dtype="f16"), 1),
    (65536, 16, 128, True, 16 * GB, dict(B=2, dtype="bf16", with_backward=True), 1),
    (1048576, 8, 128, False, 4 * GB, dict(dtype="bf16", inputs_on_device=False,
                                          acc_on_device=False), 2),
]


@pytest.mark.parametrize("L,H,d,causal,budget,kw,want", WORKLOADS)
def test_workload_depths(L, H, d, causal, budget, kw, want):
    p = cq.cqsa_plan(L, H, d, causal, budget, cq.make_opts(**kw))
    assert p.depth == want
    if budget:
        assert p.modelled_device_bytes <= budget
        if want > 1:
            # the next shallower depth must not fit (smallest feasible depth, Section 3.4)
            q = cq.cqsa_plan(L, H, d, causal, 0, cq.make_opts(depth=want - 1, **kw))
            assert q.modelled_device_bytes > budget


def _image_bytes(p, g, bwd_g=1):
    """Plan image size from the layout the planner documents: DevTask records
    (56 bytes), per-task runs, block records (OR, AND and row: 16 bytes per
    block) and the three strip orders (one int32 per strip: at bf16 d = 128
    the forward's and dQ's 256-query strips and dK/dV's 256-key strips),
    then per forward group the segments and contributions,
    and per backward launch group (when it holds several tasks) those of its
    tokens."""
    al = lambda x: (x + 255) // 256 * 256
    tasks = [p.task(t) for t in range(p.num_tasks)]
    size = al(len(tasks) * 56)
    for tk in tasks:
        nb = len(tk["block_or"])
        size += al(len(tk["runs"]) * 32) + al(nb * 16)
        size += 3 * al(-(-tk["L_local"] // 256) * 4)
    bounds = sorted({0, p.L} | {r[0] for tk in tasks for r in tk["runs"]}
                    | {r[0] + r[1] for tk in tasks for r in tk["runs"]})
    segs = list(zip(bounds[:-1], bounds[1:]))
    holders = [[t for t, tk in enumerate(tasks)
                if any(r[0] <= s0 < r[0] + r[1] for r in tk["runs"])] for s0, _ in segs]

    def groups(gs, final_all):
        n = 0
        for t0 in range(0, len(tasks), gs):
            final = final_all and t0 + gs >= len(tasks)
            n_seg = n_con = 0
            for hs in holders:
                k = sum(1 for t in hs if t0 <= t < t0 + gs)
                if k or final:
                    n_seg += 1
                    n_con += k
            n += al(n_seg * 40) + al(n_con * 16)
        return n

    size += groups(g, True)
    if bwd_g > 1:
        size += groups(bwd_g, False)
    return size


@pytest.mark.parametrize("in_place,tps,want_g,subslots",
                         [(False, 0, 1, 2), (True, 0, 7, 7)]
                         + [(ip, tps, g, n) for ip in (True, False)
                            for tps, g, n in ((1, 1, 2), (7, 7, 7), (3, 3, 6), (4, 4, 7))])
def test_footprint_model_closed_form(tps, want_g, subslots, in_place):
    """Footprint of the bf16 L=32768 H=16 d=128 depth-1 plan, recomputed here
    from the workspace layout the header documents: with g tasks per slot and
    two slots, slot i holds the largest group k = i (mod 2); a task sub-slot
    holds the statistics (acc, m, l and the rounded-weight sum lt), plus the
    staged Q, K, V unless they are read in place; with more than one launch
    group the running l and lt sit in the workspace."""
    L, H, d, B = 32768, 16, 128, 1
    p = cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(depth=1, tasks_per_slot=tps,
                                                       read_in_place=in_place))
    assert p.tasks_per_slot == want_g and p.reads_in_place == int(in_place)
    al = lambda x: (x + 255) // 256 * 256
    Lmax = max(p.task(t)["L_local"] for t in range(p.num_tasks))
    rows = B * Lmax * H
    sub = (0 if in_place else 3 * al(rows * d * 2)) + al(rows * d * 4) + 3 * al(rows * 4)
    resident = 3 * al(B * L * H * d * 2) + al(B * L * H * d * 4) + al(B * L * H * 4)
    groups = -(-7 // want_g)
    running_l = 2 * al(B * H * L * 4) if groups > 1 else 0
    want = resident + subslots * sub + running_l + al(_image_bytes(p, want_g))
    assert p.modelled_device_bytes == want


def test_backward_launch_groups():
    """Backward tasks per launch.  Inputs read in place with device-resident
    gradients and with_backward: every task (up to 32) in one dQ and one dK/dV
    launch, their task-local fp32 dQ, dK, dV (3 x B x L_max x H x d x 4 bytes
    each) counted in the backward's peak, which is then the modelled one;
    reduced until a capped budget fits.  One per launch otherwise."""
    al = lambda x: (x + 255) // 256 * 256
    L, H, d, B = 32768, 16, 128, 1
    p = cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(depth=1, with_backward=True))
    assert p.bwd_tasks_per_launch == 7
    Lmax = max(p.task(t)["L_local"] for t in range(p.num_tasks))
    f32 = al(B * L * H * d * 4)
    resident = 4 * al(B * L * H * d * 2) + f32 + al(B * H * L * 4) + 3 * f32
    local = 7 * 3 * al(B * Lmax * H * d * 4)
    want = resident + al(B * H * L * 4) + local + al(_image_bytes(p, 7, 7))
    assert p.modelled_device_bytes == want
    one = cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(depth=1, with_backward=True,
                                                       bwd_tasks_per_launch=1))
    assert one.bwd_tasks_per_launch == 1 and one.modelled_device_bytes < want
    # a budget between them: fewer tasks per launch, the same depth
    budget = (one.modelled_device_bytes + want) // 2
    mid = cq.cqsa_plan(L, H, d, False, budget, cq.make_opts(with_backward=True))
    assert mid.depth == 1 and 1 < mid.bwd_tasks_per_launch < 7
    assert mid.modelled_device_bytes <= budget
    # 49 tasks at depth 2: two launches, split evenly (25 + 24)
    p = cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(depth=2, with_backward=True))
    assert p.bwd_tasks_per_launch == 25
    # automatic sizes under a budget are balanced splits of the 7 tasks: 7, 4, 3 or 2
    for frac in (0.2, 0.4, 0.6, 0.8):
        q = cq.cqsa_plan(L, H, d, False, int(one.modelled_device_bytes + frac * (want - one.modelled_device_bytes)),
                         cq.make_opts(depth=1, with_backward=True))
        assert q.bwd_tasks_per_launch in (1, 2, 3, 4, 7), frac
    # forced
    p = cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(depth=1, with_backward=True,
                                                     bwd_tasks_per_launch=3))
    assert p.bwd_tasks_per_launch == 3
    # not batched: staged inputs, host accumulator, no with_backward, undecomposed
    for kw in (dict(read_in_place=False), dict(acc_on_device=False),
               dict(inputs_on_device=False, acc_on_device=False)):
        p = cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(depth=1, with_backward=True, **kw))
        assert p.bwd_tasks_per_launch == 1, kw
    assert cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(depth=1)).bwd_tasks_per_launch == 1
    assert cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(
        depth=0, with_backward=True)).bwd_tasks_per_launch == 1
    # refused: out of range, or forced above 1 where it cannot apply
    for kw, status in [(dict(bwd_tasks_per_launch=33), -1), (dict(bwd_tasks_per_launch=-1), -1),
                       (dict(bwd_tasks_per_launch=2, read_in_place=False), -2),
                       (dict(bwd_tasks_per_launch=2, acc_on_device=False), -2)]:
        with pytest.raises(cq.CqsaError) as e:
            cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(depth=1, with_backward=True, **kw))
        assert e.value.status == status and "bwd_tasks_per_launch" in str(e.value)


def test_group_size_rules():
    """Automatic tasks per slot.  Staged inputs: enough tasks for 1024 work
    groups per launch (128-query strips x B x H per task), capped at 32 and at
    the task count.  Inputs read in place: every task, up to 32.  One with a
    host accumulator; reduced until a capped budget fits."""
    st = dict(read_in_place=False)
    # L=4096, depth 2: 49 tasks of <= 84 tokens, 1 strip x 4 heads each
    p = cq.cqsa_plan(4096, 4, 64, False, 0, cq.make_opts(depth=2, **st))
    assert p.tasks_per_slot == 32
    # depth 1: 7 tasks of <= 586 tokens, 5 strips x 4 heads = 20 work groups each
    p = cq.cqsa_plan(4096, 4, 64, False, 0, cq.make_opts(depth=1, **st))
    assert p.tasks_per_slot == 7
    # 14043-token tasks x 16 heads: 110 x 16 = 1760 work groups, one per launch
    p = cq.cqsa_plan(32768, 16, 128, False, 0, cq.make_opts(depth=1, **st))
    assert p.tasks_per_slot == 1
    # 4682-token tasks x 16 heads: 37 x 16 = 592 -> two per launch
    p = cq.cqsa_plan(32768, 16, 128, False, 0, cq.make_opts(depth=2, **st))
    assert p.tasks_per_slot == 2
    # fp32 uses 32-query strips: 7 tasks of <= 147 tokens, 5 x 1 work groups
    p = cq.cqsa_plan(1024, 1, 64, False, 0, cq.make_opts(dtype="f32", depth=1, **st))
    assert p.tasks_per_slot == 7
    # read in place: all seven, 32 of 49
    p = cq.cqsa_plan(32768, 16, 128, False, 0, cq.make_opts(depth=1))
    assert p.reads_in_place == 1 and p.tasks_per_slot == 7
    p = cq.cqsa_plan(32768, 16, 128, False, 0, cq.make_opts(depth=2))
    assert p.tasks_per_slot == 32
    for kw in ({}, st):
        p = cq.cqsa_plan(4096, 4, 64, False, 0, cq.make_opts(depth=1, acc_on_device=False, **kw))
        assert p.tasks_per_slot == 1
        big = cq.cqsa_plan(4096, 4, 64, False, 0, cq.make_opts(depth=1, **kw))
        one = cq.cqsa_plan(4096, 4, 64, False, 0, cq.make_opts(depth=1, tasks_per_slot=1, **kw))
        budget = (big.modelled_device_bytes + one.modelled_device_bytes) // 2
        mid = cq.cqsa_plan(4096, 4, 64, False, budget, cq.make_opts(depth=1, **kw))
        assert 1 <= mid.tasks_per_slot < big.tasks_per_slot
        assert mid.modelled_device_bytes <= budget
    with pytest.raises(cq.CqsaError):
        cq.cqsa_plan(4096, 4, 64, False, 0, cq.make_opts(depth=1, tasks_per_slot=33))
    with pytest.raises(cq.CqsaError):
        cq.cqsa_plan(4096, 4, 64, False, 0, cq.make_opts(depth=1, tasks_per_slot=2,
                                                         acc_on_device=False))


def test_forward_argument_errors_without_device_work():
    torch = pytest.importorskip("torch")
    p = cq.cqsa_plan(64, 1, 64, False, 0, cq.make_opts(dtype="f32", depth=1,
                                                        inputs_on_device=False,
                                                        acc_on_device=False))
    Q = torch.zeros(1, 64, 1, 64)
    O = torch.zeros(1, 64, 1, 64)
    LSE = torch.zeros(1, 1, 64)
    bad = torch.zeros(1, 63, 1, 64)
    with pytest.raises(cq.CqsaError) as e:
        cq.cqsa_forward(p, Q, Q, bad, O, LSE)
    assert e.value.status == -1 and "shape" in str(e.value)
    with pytest.raises(cq.CqsaError) as e:
        cq.cqsa_forward(p, Q, Q, Q.half(), O, LSE)
    assert e.value.status == -1 and "dtype" in str(e.value)


def _desc(dtype, where, B=1, L=64, H=1, d=64, data=0x1000):
    """A tensor descriptor for argument checks that fail before device work
    (the data pointer is never dereferenced)."""
    code = {"f32": cq.CQSA_F32, "f16": cq.CQSA_F16, "bf16": cq.CQSA_BF16}[dtype]
    return cq.cqsa_tensor(data, code, where, B, L, H, d)


def _backward_status(plan, dt="bf16", where=None, lse=0x2000, lse_where=None, **over):
    dev = cq.CQSA_MEM_DEVICE
    where = dev if where is None else where
    t = {n: _desc(dt, where) for n in ("Q", "K", "V", "dO")}
    t.update({n: _desc("f32", where) for n in ("O", "dQ", "dK", "dV")})
    t.update(over)
    st = cq.lib().cqsa_backward(plan.handle, *(ctypes.byref(t[n]) for n in ("Q", "K", "V", "O")),
                                ctypes.c_void_p(lse), dev if lse_where is None else lse_where,
                                ctypes.byref(t["dO"]), ctypes.byref(t["dQ"]), ctypes.byref(t["dK"]),
                                ctypes.byref(t["dV"]), ctypes.c_float(0.0), ctypes.c_void_p(0))
    return st, cq.lib().cqsa_last_error().decode()


def test_backward_argument_errors_without_device_work():
    """Every argument error of cqsa_backward is reported before device work."""
    ok = cq.cqsa_plan(64, 1, 64, False, 0, cq.make_opts(depth=1, with_backward=True))
    # a capped budget fitted without the backward is refused (header contract)
    capped = cq.cqsa_plan(64, 1, 64, False, 10 ** 9, cq.make_opts(depth=1))
    st, msg = _backward_status(capped)
    assert st == -1 and "with_backward" in msg
    # fp32 plans are not built for the backward
    f32 = cq.cqsa_plan(64, 1, 64, False, 0, cq.make_opts(dtype="f32", depth=1))
    assert _backward_status(f32, dt="f32")[0] == -2
    # tensor residency, dtype and shape; LSE pointer and residency
    st, msg = _backward_status(ok, dO=_desc("bf16", cq.CQSA_MEM_HOST))
    assert st == -1 and "dO" in msg and "residency" in msg
    # a host-resident plan: inputs on the host, O, LSE and gradients too
    host = cq.cqsa_plan(64, 1, 64, False, 0, cq.make_opts(depth=1, inputs_on_device=False,
                                                          acc_on_device=False, with_backward=True))
    h = cq.CQSA_MEM_HOST
    st, msg = _backward_status(host, where=h, dQ=_desc("f32", cq.CQSA_MEM_DEVICE), lse_where=h)
    assert st == -1 and "dQ" in msg and "residency" in msg
    st, msg = _backward_status(host, where=h)
    assert st == -1 and "LSE" in msg
    st, msg = _backward_status(ok, dK=_desc("bf16", cq.CQSA_MEM_DEVICE))
    assert st == -1 and "dK" in msg and "dtype" in msg
    st, msg = _backward_status(ok, V=_desc("bf16", cq.CQSA_MEM_DEVICE, L=65))
    assert st == -1 and "V" in msg and "shape" in msg
    st, msg = _backward_status(ok, lse=0)
    assert st == -1 and "LSE" in msg
    st, msg = _backward_status(ok, lse_where=cq.CQSA_MEM_HOST)
    assert st == -1 and "LSE" in msg
    st, msg = _backward_status(ok, Q=_desc("bf16", cq.CQSA_MEM_DEVICE, data=0))
    assert st == -1 and "Q.data" in msg


def test_allocator_hook_arguments():
    with pytest.raises(ValueError):
        cq.cqsa_set_allocator(lambda n: 0, None)
    # one C function without the other is refused by the library itself
    st = cq.lib().cqsa_set_allocator(ctypes.c_void_p(0x10), None, None)
    assert st == -1 and "both" in cq.lib().cqsa_last_error().decode()
    cq.cqsa_set_allocator(None, None)   # restoring the built-in workspace is always fine


def test_out16_footprint_and_errors():
    """out16 = 1: cqsa_forward writes O in the input dtype and keeps the fp32
    result in its workspace, so the modelled peak grows by exactly the 16-bit
    O (the caller's O shrinks from fp32 to 16 bits, the workspace gains the
    fp32 copy)."""
    L, H, d = 32768, 16, 128
    for dt in ("bf16", "f16"):
        for depth in (0, 1, 2):
            a = cq.cqsa_plan(L, H, d, True, 0, cq.make_opts(dtype=dt, depth=depth))
            b = cq.cqsa_plan(L, H, d, True, 0, cq.make_opts(dtype=dt, depth=depth, out16=True))
            assert b.modelled_device_bytes - a.modelled_device_bytes == L * H * d * 2
    for kw, status in [(dict(dtype="f32", out16=True), -1),
                       (dict(out16=True, acc_on_device=False, inputs_on_device=False), -2),
                       (dict(out16=True, with_backward=True), -2)]:
        with pytest.raises(cq.CqsaError) as e:
            cq.cqsa_plan(4096, 4, 64, False, 0, cq.make_opts(**kw))
        assert e.value.status == status and "out16" in str(e.value)
    o = cq.make_opts()
    o.out16 = 2
    with pytest.raises(cq.CqsaError) as e:
        cq.cqsa_plan(4096, 4, 64, False, 0, o)
    assert e.value.status == -1


def test_out16_output_dtype_checked_before_any_device_work():
    """The O dtype must follow the plan: the input dtype with out16, fp32
    without; a mismatch is an argument error raised before any device call
    (host-resident inputs, so the tensors here never touch a GPU)."""
    B, L, H, d = 1, 256, 2, 64
    Q, K, V = (torch.zeros((B, L, H, d), dtype=torch.bfloat16) for _ in range(3))
    LSE = torch.zeros((B, H, L), dtype=torch.float32)
    for out16, odt in ((True, torch.float32), (True, torch.float16), (False, torch.bfloat16)):
        plan = cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(inputs_on_device=False, out16=out16))
        O = torch.zeros((B, L, H, d), dtype=odt)
        with pytest.raises(cq.CqsaError) as e:
            cq.cqsa_forward(plan, Q, K, V, O, LSE)
        assert e.value.status == -1 and "O has the wrong dtype" in str(e.value)


def test_misaligned_tensor_rejected_before_any_device_work():
    """Tensor data must be 16-byte aligned (rows move in 16-byte vectors): a
    contiguous view two bytes into its storage is an argument error, raised
    before any device call (host-resident tensors only)."""
    B, L, H, d = 1, 256, 2, 64
    n = B * L * H * d
    plan = cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(inputs_on_device=False))
    good = [torch.zeros((B, L, H, d), dtype=torch.bfloat16) for _ in range(2)]
    bad = torch.zeros(n + 8, dtype=torch.bfloat16)[1:1 + n].view(B, L, H, d)
    assert bad.is_contiguous() and bad.data_ptr() % 16 == 2
    O = torch.zeros((B, L, H, d), dtype=torch.float32)
    LSE = torch.zeros((B, H, L), dtype=torch.float32)
    with pytest.raises(cq.CqsaError) as e:
        cq.cqsa_forward(plan, bad, *good, O, LSE)
    assert e.value.status == -1 and "Q.data must be 16-byte aligned" in str(e.value)


def test_lse_checked_by_the_binding_before_any_call():
    """The C ABI takes LSE as a bare float pointer, so the Python binding checks
    its dtype, layout, shape (B, H, L) and residency (that of O) in both
    wrappers before calling the library: an undersized LSE would otherwise be
    written out of bounds, a bf16 or strided one misread."""
    import torch
    B, L, H, d = 2, 64, 3, 64
    plan = cq.cqsa_plan(L, H, d, False, 0, cq.make_opts(B=B, depth=1, with_backward=True))
    x = torch.zeros((B, L, H, d), dtype=torch.bfloat16)
    O = torch.zeros((B, L, H, d), dtype=torch.float32)
    good = torch.zeros((B, H, L), dtype=torch.float32)
    bad = [torch.zeros((B, H, L - 1), dtype=torch.float32),          # undersized
           torch.zeros((B, L, H), dtype=torch.float32),              # wrong layout
           torch.zeros((B, H, L), dtype=torch.bfloat16),             # wrong dtype
           torch.zeros((B, H, 2 * L), dtype=torch.float32)[..., ::2]]  # strided
    for lse in bad:
        with pytest.raises(ValueError, match="LSE"):
            cq.cqsa_forward(plan, x, x, x, O, lse)
        with pytest.raises(ValueError, match="LSE"):
            cq.cqsa_backward(plan, x, x, x, O, lse, x, O, O, O)
    # the good LSE passes the binding; the library then refuses the host
    # tensors of this device plan with a status, not a crash
    with pytest.raises(cq.CqsaError) as e:
        cq.cqsa_forward(plan, x, x, x, O, good)
    assert e.value.status == -1
