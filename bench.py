#!/usr/bin/env python3
"""Benchmark of the Stream-CQSA hot path on one MI355X.

Workload (the headline configuration): bf16 exact attention forward,
B=1, H=16, d=128, L=32768, non-causal, softmax scale 1/sqrt(d), CQS depth 1
(c=7, I=(0,1,3)), uncapped device budget, inputs/outputs device-resident.
Q, K, V are i.i.d. N(0,1) from a fixed seed, cast to bf16.

One step = one pass of the whole forward hot path: plan the call, stage every
task's runs, run the inner kernel per task (the automatic launch grouping
puts one 14043-token task in each launch here, alternating between two
compute streams), merge, finalize.  The bench also times the undecomposed
call (depth 0, one kernel) for the runtime ratio, the same forward with all
seven tasks in one launch and one merge (each kernel then runs alone, which
gives clean per-kernel rates), and the decomposed forward+backward.

`roofline` is the inner forward kernel: algorithmic FLOPs per launch over the
mean HIP-event duration of its launches in the headline run.  Consecutive
launches overlap on the two streams, so a launch shares the GPU for most of
its span; `kernels.inner_fwd` also gives the rate over the union of the
launches' spans (`achieved_busy`), the measured concurrency, and the rates of
the single-launch and undecomposed runs.

Prints one JSON line.  Algorithmic FLOPs: forward 4*d*B*H*pairs with
pairs = L^2 (non-causal); forward+backward 3.5x forward.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

B, L, H, D = 1, 32768, 16, 128
SEED = 20819 + 2
BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle sample")
    ap.add_argument("--workload", default="headline",
                    choices=["headline", "fp16_causal_L131072_8GB", "fp16_causal_L131072_8GB_c21",
                             "bf16_causal_B2_L65536_fwdbwd_16GB", "bf16_streamed_L1M_host_4GB",
                             "bf16_L32768_H16_head_dims"],
                    help="headline (default) or one of the other seeded workloads: "
                         "their rates, depths and runtime ratios, one JSON line each")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB five times (calibrates "
                         "the FETCH_SIZE / WRITE_SIZE counters) and exit")
    return ap.parse_args()


# HBM traffic of one inner forward launch, from the committed counter summary;
# reported only while the kernel sources still hash to what was profiled.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "inner_fwd_bf16_L32768_H16_d128_traffic.txt")
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


def fwd_flops(causal=False):
    pairs = L * (L + 1) // 2 if causal else L * L
    return 4.0 * D * B * H * pairs


def time_steps(step, steps, warmup, torch):
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    out = [step() for _ in range(steps)]
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / steps, out


def cpu_baseline(Q, K, V, seconds):
    """The float64 oracle on a bounded sample of query rows (all heads)."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import dense
    from paper_2604_20819_amd import synth

    Qf, Kf, Vf = synth.as_f64(Q), synth.as_f64(K), synth.as_f64(V)
    rows_per_head = 8
    done_rows, t_used = 0, 0.0
    # grow the sample until it costs about `seconds`
    while t_used < seconds and rows_per_head <= L:
        rows = synth.sample_rows(SEED, L, rows_per_head, H)
        t0 = time.perf_counter()
        dense.attention_forward(Qf, Kf, Vf, False, rows=rows)
        dt = time.perf_counter() - t0
        done_rows, t_used = rows_per_head * H, dt
        if dt * 4 > seconds:
            break
        rows_per_head *= 4
    flops = 4.0 * D * L * done_rows
    threads = sum(i.get("num_threads", 0) for i in threadpool_info()
                  if i.get("user_api") == "blas") or 1
    return {"value": flops / t_used / 1e12, "unit": "TFLOP/s", "cores": threads,
            "kind": "oracle",
            "sample": f"dense float64 forward on {done_rows // H} sampled query rows per head "
                      f"x {H} heads against all {L} keys ({t_used:.1f} s)"}


GB = 10 ** 9


def other_workload(name, args):
    """Seeded workloads beyond the headline: one JSON line each with the
    decomposed rate, the depth the budget forces, and the runtime ratio to the
    undecomposed call where that fits (host-link rates for the streamed one)."""
    import torch

    import paper_2604_20819_amd as cq
    from paper_2604_20819_amd import synth

    spec = {
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
    }[name]
    Bw, Lw, Hw, dw, causal = spec["B"], spec["L"], spec["H"], spec["d"], spec["causal"]
    host = spec["host"]
    print(f"[workload] {name}: generating inputs", file=sys.stderr, flush=True)
    ins = synth.make_inputs(spec["seed"], Bw, Lw, Hw, dw, spec["dt"], with_dO=spec["bwd"],
                            pin_memory=host)
    if host:
        q, k, v = ins[:3]
        O = torch.empty((Bw, Lw, Hw, dw), dtype=torch.float32, pin_memory=True)
        LSE = torch.empty((Bw, Hw, Lw), dtype=torch.float32, pin_memory=True)
    else:
        q, k, v = (x.cuda() for x in ins[:3])
        O = torch.empty((Bw, Lw, Hw, dw), dtype=torch.float32, device="cuda")
        LSE = torch.empty((Bw, Hw, Lw), dtype=torch.float32, device="cuda")
    pairs = Lw * (Lw + 1) // 2 if causal else Lw * Lw
    flops = 4.0 * dw * Bw * Hw * pairs

    def plan_for(depth=-1, budget=spec["budget"], backward=spec["bwd"], in_place=None):
        return cq.cqsa_plan(Lw, Hw, dw, causal, budget,
                            cq.make_opts(B=Bw, dtype=spec["dt"], depth=depth,
                                         inputs_on_device=not host, acc_on_device=not host,
                                         with_backward=backward, levels=spec.get("levels"),
                                         read_in_place=in_place))

    cq.cqsa_set_timing(True)
    steps = 2 if host else max(3, args.steps // 4)
    warm = 1

    def fwd(plan):
        def step():
            cq.cqsa_forward(plan, q, k, v, O, LSE)
            return cq.cqsa_last_stats()
        return step

    plan = plan_for()
    print(f"[workload] {name}: depth {plan.depth}, {plan.num_tasks} tasks, "
          f"{plan.tasks_per_slot} per launch", file=sys.stderr, flush=True)
    ms, st = time_steps(fwd(plan), steps, warm, torch)
    s = st[-1]
    line = {"workload": name, "B": Bw, "L": Lw, "H": Hw, "d": dw, "causal": causal,
            "dtype": spec["dt"], "budget_bytes": spec["budget"], "depth": plan.depth,
            "interest_sets": [c for c, _ in spec.get("levels", [(7, None)])],
            "tasks": plan.num_tasks, "tasks_per_launch": plan.tasks_per_slot,
            "reads_in_place": plan.reads_in_place,
            "max_task_tokens": max(task_rows(plan)),
            "task_tokens": sum(task_rows(plan)),
            "modelled_device_bytes": plan.modelled_device_bytes,
            "workspace_bytes": s["workspace_bytes"],
            # what the call holds on the device: the library's workspace plus the
            # caller's device-resident tensors (Q, K, V, O, LSE)
            "device_bytes_in_use": s["workspace_bytes"] + (0 if host else sum(
                t.numel() * t.element_size() for t in (q, k, v, O, LSE))),
            "fwd_ms": round(ms, 3), "fwd_tflops": round(flops / (ms * 1e-3) / 1e12, 2),
            "inner_fwd_busy_tflops": round(flops / (s["ms_inner_busy"] * 1e-3) / 1e12, 2)}
    if host:
        h2d, d2h = s["h2d_bytes"], s["d2h_bytes"]
        copy_ms = s["ms_stage"] + s["ms_d2h"]
        comp_ms = s["ms_inner_busy"]
        line.update({
            "h2d_bytes": h2d, "d2h_bytes": d2h,
            "h2d_GBps": round(h2d / (s["ms_stage"] * 1e-3) / 1e9, 2),
            "d2h_GBps": round(d2h / (s["ms_d2h"] * 1e-3) / 1e9, 2),
            "wall_ms": round(s["ms_wall"], 2), "compute_ms": round(comp_ms, 2),
            "copy_ms": round(copy_ms, 2), "host_merge_ms": round(s["ms_merge"], 2),
            "overlap": round(1 - (s["ms_wall"] - max(comp_ms, copy_ms)) / min(comp_ms, copy_ms), 3),
            "undecomposed": "does not apply: inputs and outputs are host-resident"})
    else:
        und = plan_for(depth=0, budget=0, backward=False)
        ms0, _ = time_steps(fwd(und), steps, warm, torch)
        line.update({"undecomposed_fwd_ms": round(ms0, 3),
                     "undecomposed_modelled_bytes": und.modelled_device_bytes,
                     "fwd_runtime_ratio": round(ms / ms0, 4)})
        # the same budget when every task's runs are gathered into staging
        # slots first: the depth it forces and its rate
        stp = plan_for(in_place=False)
        ms_s, _ = time_steps(fwd(stp), steps, warm, torch)
        line.update({"staged_depth": stp.depth, "staged_tasks": stp.num_tasks,
                     "staged_modelled_device_bytes": stp.modelled_device_bytes,
                     "staged_fwd_ms": round(ms_s, 3),
                     "staged_fwd_tflops": round(flops / (ms_s * 1e-3) / 1e12, 2)})
        if spec["bwd"]:
            do = ins[3].cuda()
            dQ, dK, dV = (torch.empty((Bw, Lw, Hw, dw), dtype=torch.float32, device="cuda")
                          for _ in range(3))

            def fb(pl):
                def step():
                    cq.cqsa_forward(pl, q, k, v, O, LSE)
                    cq.cqsa_backward(pl, q, k, v, O, LSE, do, dQ, dK, dV)
                    return cq.cqsa_last_stats()
                return step
            msb, stb = time_steps(fb(plan), steps, warm, torch)
            und_b = plan_for(depth=0, budget=0, backward=True)
            msb0, _ = time_steps(fb(und_b), steps, warm, torch)
            msb_s, _ = time_steps(fb(stp), steps, warm, torch)
            line.update({"staged_fwd_bwd_ms": round(msb_s, 3)})
            line.update({"fwd_bwd_ms": round(msb, 3),
                         "fwd_bwd_tflops": round(3.5 * flops / (msb * 1e-3) / 1e12, 2),
                         "inner_bwd_busy_tflops": round(
                             2.5 * flops / (stb[-1]["ms_inner_busy"] * 1e-3) / 1e12, 2),
                         "undecomposed_fwd_bwd_ms": round(msb0, 3),
                         "fwd_bwd_runtime_ratio": round(msb / msb0, 4)})
    cq.cqsa_set_timing(False)
    print(json.dumps(line), flush=True)


def headdim_sweep(args):
    """Forward and forward+backward rates at every head dim (32 .. 256):
    bf16, B=1 H=16 L=32768 non-causal, CQS depth 1 and undecomposed; one JSON
    line."""
    import torch

    import paper_2604_20819_amd as cq
    from paper_2604_20819_amd import synth

    B, L, H = 1, 32768, 16
    out = {"workload": "bf16_L32768_H16_head_dims", "B": B, "L": L, "H": H, "causal": False,
           "dtype": "bf16", "per_d": []}
    steps = max(3, args.steps // 4)
    for d in (32, 64, 96, 128, 160, 192, 224, 256):
        print(f"[workload] head dim {d}", file=sys.stderr, flush=True)
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


def task_rows(plan):
    return [plan.task(t)["L_local"] for t in range(plan.num_tasks)]


def main():
    args = parse()
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.workload != "headline":
        if args.gpus != 1:
            print("bench.py runs on one GPU only", file=sys.stderr)
            sys.exit(2)
        if args.workload == "bf16_L32768_H16_head_dims":
            headdim_sweep(args)
        else:
            other_workload(args.workload, args)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the decomposition shards across GPUs by design, but this build "
              "measures the single-GPU path)", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2604_20819_amd as cq
    from paper_2604_20819_amd import synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    Q, K, V, dO = synth.make_inputs(SEED, B, L, H, D, "bf16", with_dO=True)
    q, k, v, do = (x.to(dev) for x in (Q, K, V, dO))
    O = torch.empty((B, L, H, D), dtype=torch.float32, device=dev)
    LSE = torch.empty((B, H, L), dtype=torch.float32, device=dev)

    def plan_for(depth, backward=False, tps=0, in_place=None):
        return cq.cqsa_plan(L, H, D, False, 0, cq.make_opts(B=B, dtype="bf16", depth=depth,
                                                            with_backward=backward,
                                                            tasks_per_slot=tps,
                                                            read_in_place=in_place))

    def fwd_step(depth, tps=0, in_place=None, stats=True):
        def step():
            plan = plan_for(depth, tps=tps, in_place=in_place)   # planning is part of the step
            cq.cqsa_forward(plan, q, k, v, O, LSE)
            return cq.cqsa_last_stats() if stats else None
        return step

    # Each rate: steps enqueued back to back with per-stage timing off, so
    # nothing synchronises inside the timed region; then the same steps again
    # with HIP-event timing on (one synchronisation per step) for the
    # per-kernel figures.
    def rate_and_stats(depth, tps=0, in_place=None):
        cq.cqsa_set_timing(False)
        ms, _ = time_steps(fwd_step(depth, tps, in_place, stats=False), args.steps, args.warmup,
                           torch)
        cq.cqsa_set_timing(True)
        _, st = time_steps(fwd_step(depth, tps, in_place), args.steps, args.warmup, torch)
        return ms, st

    def mean(stats, key):
        return sum(s[key] for s in stats) / len(stats)

    flops = fwd_flops(False)
    # planning alone (host): part of every step below
    t0 = time.perf_counter()
    for _ in range(20):
        plan_for(1)
    plan_ms = (time.perf_counter() - t0) * 1e3 / 20
    # headline: the decomposed forward with the automatic launch grouping
    ms_dec, stats = rate_and_stats(1)
    launches = stats[-1]["inner_launches"]
    ms_launch = mean(stats, "ms_inner") / launches
    ms_busy = mean(stats, "ms_inner_busy")
    # undecomposed call (depth 0): one launch of the same kernel, no merge
    ms_und, st_und = rate_and_stats(0)
    # one task per launch on two alternating streams, merges overlapping
    ms_one, st_one = rate_and_stats(1, tps=1)
    # the same decomposition with every task's runs gathered into staging
    # slots first (the kernels otherwise read the caller's tensors in place),
    # under its own automatic grouping and in one launch
    ms_staged, st_staged = rate_and_stats(1, in_place=False)
    ms_one_st, st_one_st = rate_and_stats(1, tps=7, in_place=False)

    tflops = flops / (ms_dec * 1e-3) / 1e12
    # the seven tasks' kept pairs sum to L^2 (each pair once): flops per launch
    per_launch = flops / launches
    achieved = per_launch / (ms_launch * 1e-3) / 1e12

    plan1 = plan_for(1)
    rows = task_rows(plan1)
    pair_b = 4 * D + 8                      # acc_i row + m_i + l_i (fp32)
    merge_bytes = sum(rows) * B * H * pair_b + B * H * L * (4 * D + 4)   # one final merge
    st_all = stats if launches == 1 else st_one_st
    stage_bytes = 2 * st_one_st[-1]["d2d_bytes"]                       # read + write
    kernels = {
        "plan": {"bound": "host", "unit": "ms", "ms_per_call": round(plan_ms, 4)},
        "inner_fwd": {
            "bound": "mfma", "unit": "TFLOP/s", "launches_per_step": launches,
            "ms_per_launch": round(ms_launch, 4),
            "achieved_per_launch": round(achieved, 2),
            "concurrency": round(mean(stats, "ms_inner") / ms_busy, 3),
            "achieved_busy": round(flops / (ms_busy * 1e-3) / 1e12, 2),
            "one_task_per_launch_busy": round(flops / (mean(st_one, "ms_inner_busy") * 1e-3) / 1e12,
                                              2),
            "undecomposed_launch": round(flops / (mean(st_und, "ms_inner") * 1e-3) / 1e12, 2),
        },
        "stage": {"bound": "hbm", "unit": "GB/s", "bytes_per_step": stage_bytes,
                  "note": "staged plans only (read_in_place = 0)",
                  "achieved": round(stage_bytes / (mean(st_one_st, "ms_stage") * 1e-3) / 1e9, 1)},
        "merge_final": {"bound": "hbm", "unit": "GB/s", "bytes_per_launch": merge_bytes,
                        "note": "the single merge of an all-task launch",
                        "ms_per_launch": round(mean(st_all, "ms_merge"), 4),
                        "achieved": round(merge_bytes / (mean(st_all, "ms_merge") * 1e-3) / 1e9, 1)},
    }

    fwd_bwd = None
    try:
        dQ, dK, dV = (torch.empty((B, L, H, D), dtype=torch.float32, device=dev) for _ in range(3))
        bstats = []

        def fb_step(stats=True):
            def step():
                plan = plan_for(1, backward=True)
                cq.cqsa_forward(plan, q, k, v, O, LSE)
                cq.cqsa_backward(plan, q, k, v, O, LSE, do, dQ, dK, dV)
                if stats:
                    bstats.append(cq.cqsa_last_stats())
            return step
        cq.cqsa_set_timing(False)
        ms_fb, _ = time_steps(fb_step(False), max(3, args.steps // 2), 1, torch)
        cq.cqsa_set_timing(True)
        time_steps(fb_step(), max(3, args.steps // 2), 1, torch)
        bstats = bstats[1:]
        fwd_bwd = {"tflops": 3.5 * flops / (ms_fb * 1e-3) / 1e12, "ms_per_step": ms_fb}
        pre_bytes = B * L * H * (2 * D + 4 * D) + B * H * L * 4     # dO, O in; D out
        zero_bytes = 3 * B * L * H * D * 4
        kernels["inner_bwd"] = {
            "bound": "mfma", "unit": "TFLOP/s", "launches_per_step": bstats[-1]["inner_launches"],
            "concurrency": round(mean(bstats, "ms_inner") / mean(bstats, "ms_inner_busy"), 3),
            "achieved_busy": round(2.5 * flops / (mean(bstats, "ms_inner_busy") * 1e-3) / 1e12, 2)}
        kernels["bwd_preprocess"] = {
            "bound": "hbm", "unit": "GB/s", "bytes_per_launch": pre_bytes,
            "achieved": round(pre_bytes / (mean(bstats, "ms_finalize") * 1e-3) / 1e9, 1)}
        kernels["bwd_zero_fill"] = {
            "bound": "hbm", "unit": "GB/s", "bytes_per_step": zero_bytes,
            "achieved": round(zero_bytes / (mean(bstats, "ms_merge") * 1e-3) / 1e9, 1)}
    except cq.CqsaError as e:
        if e.status != -2:
            raise
    cq.cqsa_set_timing(False)

    line = {
        "metric": "exact attention TFLOP/s fwd & fwd+bwd vs seq len; runtime ratio vs undecomposed",
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_dec, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "bf16 exact attention forward, B=1 H=16 d=128 L=32768 "
                               "non-causal, CQS depth 1 (c=7, I=(0,1,3)), device-resident, "
                               "read in place",
                   "B": B, "H": H, "d": D, "L": L, "causal": False, "depth": 1},
        "runtime_ratio_vs_undecomposed": round(ms_dec / ms_und, 4),
        "undecomposed_ms": round(ms_und, 4),
        "undecomposed_tflops": round(flops / (ms_und * 1e-3) / 1e12, 2),
        "tasks_per_launch": stats[-1]["num_tasks"] // launches,
        "one_task_per_launch_ms": round(ms_one, 4),
        "staged_ms": round(ms_staged, 4),
        "staged_tasks_per_launch": st_staged[-1]["num_tasks"] // st_staged[-1]["inner_launches"],
        "staged_tflops": round(flops / (ms_staged * 1e-3) / 1e12, 2),
        "staged_single_launch_ms": round(ms_one_st, 4),
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / BF16_PEAK_TFLOPS, 4),
                     "traffic": measured_traffic()},
        "kernels": kernels,
    }
    if fwd_bwd is not None:
        line["fwd_bwd"] = {"tflops": round(fwd_bwd["tflops"], 2),
                           "ms_per_step": round(fwd_bwd["ms_per_step"], 4)}
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(Q, K, V, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
