#!/usr/bin/env python3
"""Benchmark of the Stream-CQSA hot path on one MI355X.

Headline (the default line): the largest single-GPU workload, a streamed
out-of-core forward -- bf16 exact attention, B=1 H=8 d=128 L=1,048,576,
non-causal, softmax scale 1/sqrt(d), Q, K, V, O and LSE in pinned host
memory, a 4 GB device budget (CQS depth 2, 49 tasks of about 192600 tokens,
accumulator on the host).  Q, K, V are i.i.d. N(0,1) from a fixed seed, cast
to bf16.  One step = one pass of the whole forward hot path: plan the call,
stage every task's runs over the host link (reusing the tokens the previous
task also holds), one inner-kernel launch per task (launches this long run
one after another on the caller's stream), copy each task's statistics back,
merge them on host threads, finalise.  `value` is algorithmic TFLOP/s = 4 d B H L^2 / step time
with the inputs already in (host) memory; the host-link rates ride along.

The same line also carries:
  * `fwd_bwd_B2_L65536`: bf16 causal B=2 H=16 d=128 L=65536 with a 16 GB
    budget (device-resident): forward and forward+backward TFLOP/s and their
    runtime ratios against the undecomposed call (depth 0);
  * `l32768`: bf16 non-causal B=1 H=16 d=128 L=32768 at depth 1
    (device-resident, read in place, all seven tasks in one launch): forward,
    forward+backward, ratios, and per-kernel rates (`kernels`);
  * `roofline`: the inner forward kernel of the headline run: algorithmic
    FLOPs per launch (the 49 tasks' kept pairs sum to L^2) over the mean
    HIP-event duration of its launches, recorded on the streams they run on;
    `inner_fwd.executed_tflops` (and `executed_*` in `kernels`) divides the
    FLOPs the products execute instead: every computed tile in full (mixed
    tiles' masked pairs included; the backward's dQ kernel recomputes S and
    dP, 14 d per pair against the algorithmic 10 d), counted from the plan's
    block summaries exactly as the kernels decide;
  * `cpu_baseline`: the float64 oracle on sampled query rows of the headline
    workload, with the rate, threads, CPU model and the extrapolated time of
    the full configuration.

Other modes (one JSON line each): --workload NAME for the seeded workloads
below, --workload sweep for the paper's shape over sequence length (fp16
causal B=1 H=8 d=64, L = 8K ... 1M: forward and forward+backward TFLOP/s and
the runtime ratio to the undecomposed call), --workload mask_skip (a CQS
task's real mask against the same task length unmasked), --workload
bf16_L32768_H16_head_dims.  Algorithmic FLOPs: forward 4 d B H pairs with
pairs = L^2 (non-causal) or L(L+1)/2 (causal); forward+backward 3.5x forward.
"""
import argparse
import gc
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_TFLOPS = 2500.0  # MI355X dense bf16 / fp16 MFMA
GB = 10 ** 9
METRIC = "exact attention TFLOP/s fwd & fwd+bwd vs seq len; runtime ratio vs undecomposed"

# Seeded workloads (seed 20819 + the workload's number).
WORKLOADS = {
    "bf16_L32768": dict(B=1, L=32768, H=16, d=128, causal=False, dt="bf16", budget=0,
                        seed=20819 + 2, host=False, bwd=True, depth=1),
    "fp16_causal_L131072_8GB": dict(B=1, L=131072, H=32, d=128, causal=True, dt="f16",
                                    budget=8 * GB, seed=20819 + 3, host=False, bwd=False),
    # the same call with the c=21 interest set (Table "interest_set"): one
    # level of 21 tasks fits the budget where c=7 needs two levels (49 tasks)
    "fp16_causal_L131072_8GB_c21": dict(B=1, L=131072, H=32, d=128, causal=True, dt="f16",
                                        budget=8 * GB, seed=20819 + 3, host=False, bwd=False,
                                        levels=[(21, (0, 1, 4, 14, 16))]),
    "bf16_causal_B2_L65536_fwdbwd_16GB": dict(B=2, L=65536, H=16, d=128, causal=True,
                                              dt="bf16", budget=16 * GB, seed=20819 + 4,
                                              host=False, bwd=True),
    "bf16_streamed_L1M_host_4GB": dict(B=1, L=1 << 20, H=8, d=128, causal=False, dt="bf16",
                                       budget=4 * GB, seed=20819 + 5, host=True, bwd=False),
    # forward+backward with every tensor in host memory (Table "recovery":
    # fwd+bwd beyond the device with the accumulator on the host)
    "bf16_streamed_L1M_host_fwdbwd_8GB": dict(B=1, L=1 << 20, H=8, d=128, causal=False,
                                              dt="bf16", budget=8 * GB, seed=20819 + 5,
                                              host=True, bwd=True),
}
HEADLINE = "bf16_streamed_L1M_host_4GB"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--headline-only", action="store_true",
                    help="time the headline workload only (no extra workloads, no CPU baseline)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle sample")
    ap.add_argument("--workload", default="headline",
                    choices=["headline", "sweep", "mask_skip", "bf16_L32768_H16_head_dims"]
                    + sorted(WORKLOADS),
                    help="headline (default) or another seeded workload, one JSON line each")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB five times (calibrates "
                         "the FETCH_SIZE / WRITE_SIZE counters) and exit")
    return ap.parse_args()


def say(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


# HBM traffic of one headline inner forward launch, from the committed
# counter summary; reported only while the kernel sources still hash to what
# was profiled.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "inner_fwd_bf16_L1M_H8_d128_streamed_traffic.txt")
KERNEL_SOURCES = ("attn_fwd.hip", "hip_common.hpp", "records.hpp", "kernels.hpp")


def kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2604_20819_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic():
    try:
        kv = dict(line.split(":", 1) for line in open(TRAFFIC_FILE) if ":" in line)
    except OSError:
        return None
    if kv.get("kernel_sources_sha256", "").strip() != kernel_source_hash():
        return None
    return int(kv["traffic_bytes_per_launch"].strip())


def copy_probe(mib):
    import torch
    n = mib * (1 << 20) // 4
    x = torch.ones(n, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(5):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": n * 4, "copy_probe_bytes_written": n * 4}))


def pairs(L, causal):
    return L * (L + 1) // 2 if causal else L * L


def time_steps(step, steps, warmup, torch):
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    out = [step() for _ in range(steps)]
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / steps, out


def warm_gpu(torch, seconds):
    """Dense fp16 products for about `seconds`, so that timing starts at
    working clocks."""
    a = torch.randn((8192, 8192), device="cuda", dtype=torch.float16)
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(10):
            a = (a @ a).clamp_(-1, 1)
        torch.cuda.synchronize()
    del a


def mean(stats, key):
    return sum(s[key] for s in stats) / len(stats)


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(Q, K, V, causal, seconds, seed):
    """The float64 oracle (dense forward) on a bounded sample: query rows of
    two heads against all keys of the workload.  Returns its rate, the threads
    it used, the CPU, and the extrapolated time of the full configuration."""
    from threadpoolctl import threadpool_info

    from oracle import dense
    from paper_2604_20819_amd import synth

    B, L, H, d = Q.shape
    heads = sorted({0, H // 2})
    # per-head float32 copies (exact for 16-bit inputs); the oracle converts
    # to float64 itself
    arr = {h: tuple(x[:, :, h:h + 1].float().numpy() for x in (Q, K, V)) for h in heads}
    n = 8
    while True:
        rows = synth.sample_rows(seed, L, n, H)
        t_used = 0.0
        for h in heads:
            t0 = time.perf_counter()
            dense.attention_forward(*arr[h], causal, rows=[rows[h]])
            t_used += time.perf_counter() - t0
        # stop once the sample costs about `seconds` (the next doubling would
        # overshoot it)
        if t_used * 2.5 > seconds or n >= L:
            break
        n *= 2
    keys = sum(int(r) + 1 if causal else L for h in heads for r in rows[h]) * B
    rate = 4.0 * d * keys / t_used
    full = 4.0 * d * B * H * pairs(L, causal)
    threads = sum(i.get("num_threads", 0) for i in threadpool_info()
                  if i.get("user_api") == "blas") or 1
    return {"value": round(rate / 1e12, 6), "unit": "TFLOP/s", "cores": threads,
            "kind": "oracle",
            "sample": f"dense float64 forward on {n} sampled query rows of each of heads "
                      f"{heads} against all {L} keys ({t_used:.1f} s of oracle time)",
            "cpu_model": cpu_model(), "host_cpus": len(os.sched_getaffinity(0)),
            "extrapolated_full_config_s": round(full / rate, 1)}


def make_workload(spec, torch, synth, with_dO=None):
    """Seeded inputs (pinned host or device) and outputs of a workload."""
    Bw, Lw, Hw, dw = spec["B"], spec["L"], spec["H"], spec["d"]
    host = spec["host"]
    bwd = spec["bwd"] if with_dO is None else with_dO
    ins = synth.make_inputs(spec["seed"], Bw, Lw, Hw, dw, spec["dt"], with_dO=bwd,
                            pin_memory=host)
    if host:
        dev = list(ins)
        mk = lambda *s: torch.empty(s, dtype=torch.float32, pin_memory=True)
    else:
        dev = [x.cuda() for x in ins]
        mk = lambda *s: torch.empty(s, dtype=torch.float32, device="cuda")
    return ins, dev, mk


def plan_for(cq, spec, depth=-1, budget=None, backward=None, in_place=None, tps=0):
    return cq.cqsa_plan(spec["L"], spec["H"], spec["d"], spec["causal"],
                        spec["budget"] if budget is None else budget,
                        cq.make_opts(B=spec["B"], dtype=spec["dt"], depth=depth,
                                     inputs_on_device=not spec["host"],
                                     acc_on_device=not spec["host"],
                                     with_backward=spec["bwd"] if backward is None else backward,
                                     levels=spec.get("levels"), read_in_place=in_place,
                                     tasks_per_slot=tps))


def streamed_figures(s):
    """Host-link figures of one streamed call's stats (PCIe-inclusive)."""
    h2d, d2h = s["h2d_bytes"], s["d2h_bytes"]
    copy_ms = s["ms_stage"] + s["ms_d2h"]
    comp_ms = s["ms_inner_busy"]
    return {"h2d_bytes": h2d, "d2h_bytes": d2h, "d2d_reuse_bytes": s["d2d_bytes"],
            "h2d_GBps": round(h2d / (s["ms_stage"] * 1e-3) / 1e9, 2) if s["ms_stage"] else None,
            "d2h_GBps": round(d2h / (s["ms_d2h"] * 1e-3) / 1e9, 2) if s["ms_d2h"] else None,
            "wall_ms": round(s["ms_wall"], 2), "compute_ms": round(comp_ms, 2),
            "copy_ms": round(copy_ms, 2), "host_merge_ms": round(s["ms_merge"], 2),
            "overlap": round(1 - (s["ms_wall"] - max(comp_ms, copy_ms)) / min(comp_ms, copy_ms), 3)
            if min(comp_ms, copy_ms) > 0 else None}


def run_workload(name, steps, warmup):
    """One seeded workload: the decomposed forward's rate and depth, the
    runtime ratio to the undecomposed call where it fits, the staged plan
    under the same budget, and forward+backward where the workload has it."""
    import torch

    import paper_2604_20819_amd as cq
    from paper_2604_20819_amd import synth

    spec = WORKLOADS[name]
    Bw, Lw, Hw, dw, causal, host = (spec[k] for k in ("B", "L", "H", "d", "causal", "host"))
    say(f"{name}: generating inputs")
    ins, (q, k, v, *rest), mk = make_workload(spec, torch, synth)
    O, LSE = mk(Bw, Lw, Hw, dw), mk(Bw, Hw, Lw)
    flops = 4.0 * dw * Bw * Hw * pairs(Lw, causal)
    depth = spec.get("depth", -1)

    def fwd(plan):
        def step():
            cq.cqsa_forward(plan, q, k, v, O, LSE)
            return cq.cqsa_last_stats()
        return step

    cq.cqsa_set_timing(True)
    plan = plan_for(cq, spec, depth=depth)
    say(f"{name}: depth {plan.depth}, {plan.num_tasks} tasks, {plan.tasks_per_slot} per launch")
    ms, st = time_steps(fwd(plan), steps, warmup, torch)
    s = st[-1]
    rows = [plan.task(t)["L_local"] for t in range(plan.num_tasks)]
    line = {"workload": name, "B": Bw, "L": Lw, "H": Hw, "d": dw, "causal": causal,
            "dtype": spec["dt"], "budget_bytes": spec["budget"], "depth": plan.depth,
            "interest_sets": [c for c, _ in spec.get("levels", [(7, None)])],
            "tasks": plan.num_tasks, "tasks_per_launch": plan.tasks_per_slot,
            "reads_in_place": plan.reads_in_place, "max_task_tokens": max(rows),
            "task_tokens": sum(rows), "modelled_device_bytes": plan.modelled_device_bytes,
            "workspace_bytes": s["workspace_bytes"],
            "fwd_ms": round(ms, 3), "fwd_tflops": round(flops / (ms * 1e-3) / 1e12, 2),
            "inner_fwd_busy_tflops": round(flops / (mean(st, "ms_inner_busy") * 1e-3) / 1e12, 2)}
    if host:
        line.update(streamed_figures(s))
        line["undecomposed"] = "does not apply: inputs and outputs are host-resident"
    else:
        und = plan_for(cq, spec, depth=0, budget=0, backward=False)
        ms0, _ = time_steps(fwd(und), steps, warmup, torch)
        line.update({"undecomposed_fwd_ms": round(ms0, 3),
                     "undecomposed_fwd_tflops": round(flops / (ms0 * 1e-3) / 1e12, 2),
                     "fwd_runtime_ratio": round(ms / ms0, 4)})
        if spec["budget"]:
            # the same budget when every task's runs are gathered into
            # staging slots first: the depth it forces and its rate
            stp = plan_for(cq, spec, depth=depth, in_place=False)
            ms_s, _ = time_steps(fwd(stp), steps, warmup, torch)
            line.update({"staged_depth": stp.depth, "staged_tasks": stp.num_tasks,
                         "staged_modelled_device_bytes": stp.modelled_device_bytes,
                         "staged_fwd_ms": round(ms_s, 3),
                         "staged_fwd_tflops": round(flops / (ms_s * 1e-3) / 1e12, 2)})
    if spec["bwd"]:
        do = rest[0]
        dQ, dK, dV = mk(Bw, Lw, Hw, dw), mk(Bw, Lw, Hw, dw), mk(Bw, Lw, Hw, dw)

        def fb(pl):
            def step():
                cq.cqsa_forward(pl, q, k, v, O, LSE)
                cq.cqsa_backward(pl, q, k, v, O, LSE, do, dQ, dK, dV)
                return cq.cqsa_last_stats()
            return step
        msb, stb = time_steps(fb(plan), steps, warmup, torch)
        line.update({"fwd_bwd_ms": round(msb, 3),
                     "fwd_bwd_tflops": round(3.5 * flops / (msb * 1e-3) / 1e12, 2),
                     "inner_bwd_busy_tflops": round(
                         2.5 * flops / (mean(stb, "ms_inner_busy") * 1e-3) / 1e12, 2)})
        if host:
            line["bwd_streamed"] = streamed_figures(stb[-1])
        else:
            und_b = plan_for(cq, spec, depth=0, budget=0, backward=True)
            msb0, _ = time_steps(fb(und_b), steps, warmup, torch)
            line.update({"undecomposed_fwd_bwd_ms": round(msb0, 3),
                         "undecomposed_fwd_bwd_tflops": round(3.5 * flops / (msb0 * 1e-3) / 1e12, 2),
                         "fwd_bwd_runtime_ratio": round(msb / msb0, 4)})
    cq.cqsa_set_timing(False)
    return line


def l32768_kernels(steps, warmup):
    """Per-kernel rates of the bf16 L=32768 H=16 d=128 depth-1 call (inner
    forward per launch, the all-task merge, the staged gather, the backward's
    kernels, preprocess and gradient merge); each kernel measured while it
    runs alone on the GPU."""
    import torch

    import paper_2604_20819_amd as cq

    from paper_2604_20819_amd import synth
    spec = WORKLOADS["bf16_L32768"]
    B, L, H, D = spec["B"], spec["L"], spec["H"], spec["d"]
    ins, (q, k, v, do), mk = make_workload(spec, torch, synth)
    O, LSE = mk(B, L, H, D), mk(B, H, L)
    flops = 4.0 * D * B * H * L * L
    cq.cqsa_set_timing(True)

    def fstep(plan):
        def step():
            cq.cqsa_forward(plan, q, k, v, O, LSE)
            return cq.cqsa_last_stats()
        return step
    plan = plan_for(cq, spec, depth=1)
    _, st = time_steps(fstep(plan), steps, warmup, torch)
    launches = st[-1]["inner_launches"]
    ms_launch = mean(st, "ms_inner") / launches
    rows = [plan.task(t)["L_local"] for t in range(plan.num_tasks)]
    merge_bytes = sum(rows) * B * H * (4 * D + 12) + B * H * L * (4 * D + 4)
    stp = plan_for(cq, spec, depth=1, in_place=False, tps=7)
    _, sts = time_steps(fstep(stp), steps, warmup, torch)
    stage_bytes = 2 * sts[-1]["d2d_bytes"]
    und = plan_for(cq, spec, depth=0)
    _, stu = time_steps(fstep(und), steps, warmup, torch)
    dQ, dK, dV = mk(B, L, H, D), mk(B, L, H, D), mk(B, L, H, D)

    def fb():
        cq.cqsa_forward(plan, q, k, v, O, LSE)
        cq.cqsa_backward(plan, q, k, v, O, LSE, do, dQ, dK, dV)
        return cq.cqsa_last_stats()
    _, stb = time_steps(fb, steps, warmup, torch)
    cq.cqsa_set_timing(False)
    pre_bytes = B * L * H * (2 * D + 4 * D) + B * H * L * 4
    # the backward's gradient merge (all seven tasks in one launch group):
    # every task's local dQ, dK, dV rows read once, the gradients written once
    gmerge_bytes = 3 * (sum(rows) + L) * B * H * D * 4
    return {
        "inner_fwd": {"bound": "mfma", "unit": "TFLOP/s", "launches_per_step": launches,
                      "ms_per_launch": round(ms_launch, 4),
                      "achieved_per_launch": round(flops / launches / (ms_launch * 1e-3) / 1e12, 2),
                      "executed_tflops_per_launch": round(
                          fwd_executed_flops(plan, D) / launches / (ms_launch * 1e-3) / 1e12, 2),
                      "frac": round(flops / launches / (ms_launch * 1e-3) / 1e12 / PEAK_TFLOPS, 4),
                      "undecomposed_launch": round(
                          flops / (mean(stu, "ms_inner") * 1e-3) / 1e12, 2)},
        "merge_final": {"bound": "hbm", "unit": "GB/s", "bytes_per_launch": merge_bytes,
                        "ms_per_launch": round(mean(st, "ms_merge"), 4),
                        "achieved": round(merge_bytes / (mean(st, "ms_merge") * 1e-3) / 1e9, 1)},
        "stage": {"bound": "hbm", "unit": "GB/s", "bytes_per_step": stage_bytes,
                  "note": "staged plans only (read_in_place = 0)",
                  "achieved": round(stage_bytes / (mean(sts, "ms_stage") * 1e-3) / 1e9, 1)},
        "inner_bwd": {"bound": "mfma", "unit": "TFLOP/s",
                      "launches_per_step": stb[-1]["inner_launches"],
                      "concurrency": round(mean(stb, "ms_inner") / mean(stb, "ms_inner_busy"), 3),
                      "achieved_busy": round(
                          2.5 * flops / (mean(stb, "ms_inner_busy") * 1e-3) / 1e12, 2),
                      "frac": round(2.5 * flops / (mean(stb, "ms_inner_busy") * 1e-3) / 1e12
                                    / PEAK_TFLOPS, 4),
                      "executed_busy": round(
                          bwd_executed_flops(plan, D) / (mean(stb, "ms_inner_busy") * 1e-3) / 1e12,
                          2)},
        "bwd_preprocess": {"bound": "hbm", "unit": "GB/s", "bytes_per_launch": pre_bytes,
                           "achieved": round(pre_bytes / (mean(stb, "ms_finalize") * 1e-3) / 1e9,
                                             1)},
        "bwd_grad_merge": {"bound": "hbm", "unit": "GB/s", "bytes_per_launch": gmerge_bytes,
                           "launches_per_step": stb[-1]["merge_launches"],
                           "achieved": round(gmerge_bytes / (mean(stb, "ms_merge") * 1e-3) / 1e9,
                                             1)},
    }


def sweep(args):
    """The paper's shape (Sec. 4.1: causal, B=1, H=8, D=64, fp16) over sequence
    length: the decomposed call at depth 1 (the paper's itr=1) and the
    undecomposed call, forward and forward+backward, device-resident."""
    import torch

    import paper_2604_20819_amd as cq
    from paper_2604_20819_amd import synth

    B, H, d = 1, 8, 64
    out = {"workload": "sweep_fp16_causal_B1_H8_d64", "B": B, "H": H, "d": d, "causal": True,
           "dtype": "f16", "depth": 1, "per_L": []}
    for L in [8192 << i for i in range(8)]:
        say(f"sweep L={L}")
        Q, K, V, dO = synth.make_inputs(20819 + 100 + L.bit_length(), B, L, H, d, "f16",
                                        with_dO=True)
        q, k, v, do = (x.cuda() for x in (Q, K, V, dO))
        O = torch.empty((B, L, H, d), dtype=torch.float32, device="cuda")
        LSE = torch.empty((B, H, L), dtype=torch.float32, device="cuda")
        dQ, dK, dV = (torch.empty((B, L, H, d), dtype=torch.float32, device="cuda")
                      for _ in range(3))
        flops = 4.0 * d * B * H * pairs(L, True)
        # short calls take more steps, and a second of warm-up work before the
        # first length brings the GPU's clocks up (the first sub-millisecond
        # calls of a process otherwise run up to 1.7x slower)
        steps = 20 if L <= (1 << 15) else 5 if L <= (1 << 17) else 2
        if L == 8192:
            warm_gpu(torch, 1.0)
        row = {"L": L}
        for depth, tag in ((1, "decomposed"), (0, "undecomposed")):
            plan = cq.cqsa_plan(L, H, d, True, 0, cq.make_opts(B=B, dtype="f16", depth=depth,
                                                                with_backward=True))
            ms, _ = time_steps(lambda: cq.cqsa_forward(plan, q, k, v, O, LSE), steps, 3, torch)

            def fb():
                cq.cqsa_forward(plan, q, k, v, O, LSE)
                cq.cqsa_backward(plan, q, k, v, O, LSE, do, dQ, dK, dV)
            msb, _ = time_steps(fb, steps, 3, torch)
            row.update({f"{tag}_fwd_ms": round(ms, 3),
                        f"{tag}_fwd_tflops": round(flops / (ms * 1e-3) / 1e12, 2),
                        f"{tag}_fwd_bwd_ms": round(msb, 3),
                        f"{tag}_fwd_bwd_tflops": round(3.5 * flops / (msb * 1e-3) / 1e12, 2)})
        row["fwd_runtime_ratio"] = round(row["decomposed_fwd_ms"] / row["undecomposed_fwd_ms"], 4)
        row["fwd_bwd_runtime_ratio"] = round(
            row["decomposed_fwd_bwd_ms"] / row["undecomposed_fwd_bwd_ms"], 4)
        out["per_L"].append(row)
        del q, k, v, do, O, LSE, dQ, dK, dV
        torch.cuda.empty_cache()
    print(json.dumps(out), flush=True)


def mask_skip(args):
    """App. A.2 ("Skipping fully-masked tiles"): a depth-2 task of the paper's
    N = 262144 causal fp16 shape (H=8, d=64) with its real CQS mask, whose
    fully masked tiles are skipped, against a causal attention call of the
    same length with no CQS mask (every causally live tile computed).  Each
    task's launch is timed alone (one slot, one task per launch)."""
    import torch

    import paper_2604_20819_amd as cq
    from paper_2604_20819_amd import synth

    B, L, H, d = 1, 262144, 8, 64
    Q, K, V = synth.make_inputs(20819 + 7, B, L, H, d, "f16")
    q, k, v = (x.cuda() for x in (Q, K, V))
    O = torch.empty((B, L, H, d), dtype=torch.float32, device="cuda")
    LSE = torch.empty((B, H, L), dtype=torch.float32, device="cuda")
    plan = cq.cqsa_plan(L, H, d, True, 0, cq.make_opts(B=B, dtype="f16", depth=2, n_slots=1,
                                                        tasks_per_slot=1))
    cq.cqsa_set_timing(True)
    _, st = time_steps(lambda: (cq.cqsa_forward(plan, q, k, v, O, LSE), cq.cqsa_last_stats())[1],
                       max(2, args.steps), 1, torch)
    task_ms = mean(st, "ms_inner") / st[-1]["inner_launches"]
    rows = [plan.task(t)["L_local"] for t in range(plan.num_tasks)]
    Li = int(round(sum(rows) / len(rows)))
    q2, k2, v2 = q[:, :Li].contiguous(), k[:, :Li].contiguous(), v[:, :Li].contiguous()
    O2 = torch.empty((B, Li, H, d), dtype=torch.float32, device="cuda")
    LSE2 = torch.empty((B, H, Li), dtype=torch.float32, device="cuda")
    und = cq.cqsa_plan(Li, H, d, True, 0, cq.make_opts(B=B, dtype="f16", depth=0))
    _, st2 = time_steps(lambda: (cq.cqsa_forward(und, q2, k2, v2, O2, LSE2),
                                 cq.cqsa_last_stats())[1], max(2, args.steps), 1, torch)
    cq.cqsa_set_timing(False)
    full, clear, mixed = plan.tile_census()
    tot = full + clear + mixed
    print(json.dumps({
        "workload": "mask_skip_fp16_causal_L262144_H8_d64_depth2", "tasks": plan.num_tasks,
        "mean_task_tokens": Li, "real_mask_task_launch_ms": round(task_ms, 4),
        "unmasked_same_length_ms": round(mean(st2, "ms_inner"), 4),
        "speedup_from_skipping": round(mean(st2, "ms_inner") / task_ms, 3),
        "census_pct": {"fully_masked": round(100 * full / tot, 2),
                       "clear": round(100 * clear / tot, 2), "mixed": round(100 * mixed / tot, 2)},
        "ideal_speedup": round(tot / (clear + mixed), 3)}), flush=True)


def headdim_sweep(args):
    """Forward and forward+backward rates at every head dim (32 .. 256):
    bf16, B=1 H=16 L=32768 non-causal, CQS depth 1 and undecomposed."""
    import torch

    import paper_2604_20819_amd as cq
    from paper_2604_20819_amd import synth

    B, L, H = 1, 32768, 16
    out = {"workload": "bf16_L32768_H16_head_dims", "B": B, "L": L, "H": H, "causal": False,
           "dtype": "bf16", "per_d": []}
    steps = max(3, args.steps)
    for d in (32, 64, 96, 128, 160, 192, 224, 256):
        say(f"head dim {d}")
        Q, K, V, dO = synth.make_inputs(20819 + d, B, L, H, d, "bf16", with_dO=True)
        q, k, v, do = (x.cuda() for x in (Q, K, V, dO))
        O = torch.empty((B, L, H, d), dtype=torch.float32, device="cuda")
        LSE = torch.empty((B, H, L), dtype=torch.float32, device="cuda")
        dQ, dK, dV = (torch.empty((B, L, H, d), dtype=torch.float32, device="cuda") for _ in range(3))
        flops = 4.0 * d * B * H * L * L
        row = {"d": d}
        for depth in (1, 0):
            plan = cq.cqsa_plan(L, H, d, False, 0,
                                cq.make_opts(B=B, dtype="bf16", depth=depth, with_backward=True))
            ms, _ = time_steps(lambda: cq.cqsa_forward(plan, q, k, v, O, LSE), steps, 1, torch)
            tag = "depth1" if depth else "undecomposed"
            row[tag + "_tflops"] = round(flops / (ms * 1e-3) / 1e12, 2)
            row[tag + "_ms"] = round(ms, 3)

            def fb():
                cq.cqsa_forward(plan, q, k, v, O, LSE)
                cq.cqsa_backward(plan, q, k, v, O, LSE, do, dQ, dK, dV)
            msb, _ = time_steps(fb, max(3, steps // 2), 2, torch)
            row[tag + "_fwd_bwd_tflops"] = round(3.5 * flops / (msb * 1e-3) / 1e12, 2)
            row[tag + "_fwd_bwd_ms"] = round(msb, 3)
        row["fwd_runtime_ratio"] = round(row["depth1_ms"] / row["undecomposed_ms"], 4)
        row["fwd_bwd_runtime_ratio"] = round(row["depth1_fwd_bwd_ms"] / row["undecomposed_fwd_bwd_ms"], 4)
        out["per_d"].append(row)
        del q, k, v, do, O, LSE, dQ, dK, dV
        torch.cuda.empty_cache()
    print(json.dumps(out), flush=True)


def fwd_executed_flops(plan, D):
    """FLOPs the inner forward's products execute: 4 D per (query, key) pair of
    every 32-query x 64-key wave tile it computes (clear or mixed), counted by
    the plan's block summaries exactly as the kernel decides (the kernel's own
    counters equal these counts, tests/test_gpu_tile_counts.py)."""
    _, clear, mixed = plan.fwd_tile_decisions()
    return (clear + mixed) * 32 * 64 * 4.0 * D


def bwd_executed_flops(plan, D):
    """FLOPs the backward kernels' products execute: dQ 6 D per pair of its
    computed 32-query x 64-key wave tiles (S, dP, dQ), dK/dV 8 D per pair of
    its computed 32-key x T-query tiles (S, dP, dV, dK; T from
    cqsa_bwd_kv_query_tile)."""
    import paper_2604_20819_amd as cq

    (_, qc, qm), (_, kc, km) = plan.bwd_tile_decisions()
    t = cq.cqsa_bwd_kv_query_tile(D)
    return (qc + qm) * 32 * 64 * 6.0 * D + (kc + km) * 32 * t * 8.0 * D


def headline(args):
    import torch

    import paper_2604_20819_amd as cq
    from paper_2604_20819_amd import synth

    spec = WORKLOADS[HEADLINE]
    B, L, H, D = spec["B"], spec["L"], spec["H"], spec["d"]
    say("headline: generating inputs in pinned host memory")
    ins, (q, k, v), mk = make_workload(spec, torch, synth)
    O, LSE = mk(B, L, H, D), mk(B, H, L)
    flops = 4.0 * D * B * H * L * L

    def step():
        plan = plan_for(cq, spec)          # planning is part of the step
        cq.cqsa_forward(plan, q, k, v, O, LSE)
        return cq.cqsa_last_stats(), plan

    # HIP-event timing on: the call blocks on its host-resident outputs
    # anyway, so the events add no synchronisation to the timed steps
    cq.cqsa_set_timing(True)
    say(f"headline: {args.warmup} warmup + {args.steps} timed steps")
    ms, out = time_steps(step, args.steps, args.warmup, torch)
    cq.cqsa_set_timing(False)
    st = [s for s, _ in out]
    plan = out[-1][1]
    launches = st[-1]["inner_launches"]
    ms_launch = mean(st, "ms_inner") / launches
    per_launch = flops / launches          # the tasks' kept pairs sum to L^2
    achieved = per_launch / (ms_launch * 1e-3) / 1e12
    executed = fwd_executed_flops(plan, D) / launches
    line = {
        "metric": METRIC,
        "value": round(flops / (ms * 1e-3) / 1e12, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "streamed out-of-core bf16 exact attention forward, B=1 H=8 "
                               "d=128 L=1048576 non-causal, Q/K/V/O/LSE in pinned host memory, "
                               "4 GB device budget (CQS depth 2, c=7, I=(0,1,3), 49 tasks, "
                               "accumulator on the host)",
                   "B": B, "H": H, "d": D, "L": L, "causal": False, "depth": plan.depth,
                   "tasks": plan.num_tasks, "budget_bytes": spec["budget"],
                   "modelled_device_bytes": plan.modelled_device_bytes,
                   "workspace_bytes": st[-1]["workspace_bytes"]},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_TFLOPS, 4),
                     "traffic": measured_traffic()},
        "inner_fwd": {"kernel": "attn_fwd_mfma<BF16, 128, stats>", "launches_per_step": launches,
                      "flops_per_launch": per_launch, "ms_per_launch": round(ms_launch, 4),
                      "executed_flops_per_launch": executed,
                      "executed_tflops": round(executed / (ms_launch * 1e-3) / 1e12, 2),
                      "concurrency": round(mean(st, "ms_inner") / mean(st, "ms_inner_busy"), 3),
                      "achieved_busy": round(flops / (mean(st, "ms_inner_busy") * 1e-3) / 1e12,
                                             2)},
        "streamed": streamed_figures(st[-1]),
    }
    if not args.no_cpu_baseline and not args.headline_only:
        say("headline: CPU baseline (float64 oracle on sampled rows)")
        line["cpu_baseline"] = cpu_baseline(ins[0], ins[1], ins[2], False, args.cpu_seconds,
                                            spec["seed"])
    del ins, q, k, v, O, LSE
    gc.collect()
    if not args.headline_only:
        extra_steps = max(3, args.steps // 4)
        w = run_workload("bf16_causal_B2_L65536_fwdbwd_16GB", extra_steps, 1)
        line["fwd_bwd_B2_L65536"] = {k: w[k] for k in (
            "workload", "depth", "tasks", "fwd_tflops", "fwd_runtime_ratio", "fwd_bwd_tflops",
            "fwd_bwd_ms", "undecomposed_fwd_bwd_ms", "fwd_bwd_runtime_ratio",
            "inner_bwd_busy_tflops")}
        gc.collect()
        torch.cuda.empty_cache()
        w = run_workload("bf16_L32768", max(5, args.steps // 2), 2)
        line["l32768"] = {k: w[k] for k in (
            "workload", "depth", "fwd_ms", "fwd_tflops", "undecomposed_fwd_ms",
            "fwd_runtime_ratio", "fwd_bwd_ms", "fwd_bwd_tflops", "undecomposed_fwd_bwd_ms",
            "fwd_bwd_runtime_ratio")}
        line["kernels"] = l32768_kernels(max(5, args.steps // 2), 2)
    print(json.dumps(line), flush=True)


def main():
    args = parse()
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported (the "
              "decomposition shards across GPUs by design, but this build measures the "
              "single-GPU path)", file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    if args.workload == "headline":
        headline(args)
    elif args.workload == "sweep":
        sweep(args)
    elif args.workload == "mask_skip":
        mask_skip(args)
    elif args.workload == "bf16_L32768_H16_head_dims":
        headdim_sweep(args)
    else:
        print(json.dumps(run_workload(args.workload, max(2, args.steps), 1)), flush=True)


if __name__ == "__main__":
    main()
