#!/usr/bin/env python3
"""Benchmark: Tree-LSTM fwd+bwd vertices/sec (h=512, batch 256) on one MI355X.

A step is one pass of the whole path over one batch of synthetic parse-shaped
trees (child-sum Tree-LSTM, D=300, H=512, 256 trees, CE loss at every vertex):
cavs_schedule (level assignment + level-major compaction), cavs_forward
(pull GEMM, per-level fused gather/GEMM/gates, loss head) and cavs_backward
(per-level gates + GEMM with child scatter, lazy weight gradients).  Inputs
are resident in HBM before the timed region.

Prints one JSON line with the throughput, a roofline entry for the kernel
that takes the most time (per-launch algorithmic FLOPs over its mean launch
duration, from HIP events on the library's stream) and the CPU oracle timed
on a bounded sample of the same workload.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "Tree-LSTM fwd+bwd vertices/sec (h=512, batch 256); % MFMA / HBM roofline"
PEAK_FP32_TFLOPS = 157.3     # MI355X dense fp32 matrix
PEAK_HBM_GBS = 8000.0        # MI355X HBM3E


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-trees", type=int, default=48,
                    help="graphs in the CPU-oracle sample (0 skips the CPU baseline)")
    return ap.parse_args()


def algorithmic_costs(wl, sh, n_pull, with_f):
    """Algorithmic FLOPs (and bytes for elementwise kernels) per kernel name
    for one step, from the schedule.  Only work the method must do counts:
    absent children and unused gate blocks contribute nothing."""
    import numpy as np
    H, D, N = wl.H, wl.D, wl.N
    lo = sh["level_offsets"]
    cp = sh["child_pos"].reshape(-1, N)
    nc = (cp >= 0).sum(axis=1)
    costs = {}

    def add(name, flops=0.0, nbytes=0.0):
        f, b = costs.get(name, (0.0, 0.0))
        costs[name] = (f + flops, b + nbytes)

    T = sh["T"]
    for t in range(T):
        a, b = int(lo[t]), int(lo[t + 1])
        M = b - a
        if wl.cell == 0:
            if t == 0:
                add("k_lstm_leaf", 0.0, M * H * 4.0 * 12)
                add("k_lstm_bwd_gates", 0.0, M * H * 4.0 * 12)
                continue
            fl = float(np.sum(2.0 * H * (3 * H + nc[a:b] * H)))
            v = 16 if M <= 32 else 64
            add("k_lstm_fwd_level<%d, %d>" % (N, v), fl)
            add("k_lstm_bwd_level<%d, %d>" % (N, v), fl)
            add("k_lstm_bwd_gates", 0.0, M * H * 4.0 * (10 + 3 * N))
        else:
            if t == 0:
                continue
            fl = float(np.sum(2.0 * nc[a:b] * H * H))
            v = 16 if M <= 32 else 64
            add("k_fc_fwd_level<%d>" % v, fl)
            add("k_fc_bwd_level<%d>" % v, fl)
    inner = nc > 0
    if wl.cell == 0:
        gates_x = 4 if with_f else 3
        add("k_pull_gemm", 2.0 * n_pull * D * gates_x * H)
        add("k_dx_gemm", 2.0 * n_pull * D * gates_x * H)
        add("k_tn_gemm<LdDWx>", 2.0 * n_pull * D * gates_x * H)
        if N == 2:
            add("k_tn_gemm<LdDUiou>", 2.0 * H * 3 * H * int(inner.sum()))
            add("k_tn_gemm<LdDUf>", 2.0 * H * H * float(nc.sum()))
        else:
            add("k_tn_gemm<LdDUiou>", 2.0 * H * 4 * H * int(inner.sum()))
    else:
        add("k_tn_gemm<LdFCdW>", 2.0 * H * H * float(nc.sum()))
    return costs


def cpu_baseline(wl, n_trees):
    """The oracle as it stands (fp64, recursive, one thread) on the first
    n_trees graphs of the batch."""
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import oracle
    from parity import subset
    n_trees = min(n_trees, wl.K)
    sub = subset(wl, list(range(n_trees)))
    oracle.lib()
    t0 = time.perf_counter()
    oracle.run(sub)
    dt = time.perf_counter() - t0
    return {"value": sub.V / dt, "unit": "vertices/s", "cores": 1, "kind": "oracle",
            "sample": "first %d of %d graphs (%d of %d vertices), fp64 recursive oracle, "
                      "forward + loss + backward, one thread, %.1f s"
                      % (n_trees, wl.K, sub.V, wl.V, dt)}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only (the path has no multi-GPU component in this "
              "build); got --gpus %d, WORLD_SIZE=%d" % (args.gpus, world), file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_1712_04048_amd import binding as B
    from paper_1712_04048_amd import workloads as W
    from paper_1712_04048_amd.runner import Batch

    torch.cuda.set_device(0)
    wl = W.config_treelstm_sst(args.seed)
    ctx = B.Context(0)
    batch = Batch(wl, ctx)
    batch.schedule()
    batch.alloc()
    stream = torch.cuda.current_stream()

    for _ in range(args.warmup):
        batch.step()
    torch.cuda.synchronize()

    # timed region: K whole steps (schedule + forward + backward)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        batch.step()
    ev1.record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    wall_ms = (t1 - t0) * 1e3 / args.steps
    gpu_ms = ev0.elapsed_time(ev1) / args.steps

    # breakdown: schedule alone, forward+backward alone
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for _ in range(args.steps):
        batch.schedule()
    torch.cuda.synchronize()
    sched_ms = (time.perf_counter() - t2) * 1e3 / args.steps
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        batch.forward()
        batch.backward()
    e1.record(stream)
    torch.cuda.synchronize()
    fwdbwd_ms = e0.elapsed_time(e1) / args.steps

    # per-kernel durations: the same steps again with per-launch HIP events
    ctx.timing(True)
    for _ in range(args.steps):
        batch.step()
    times = ctx.timing_read()
    ctx.timing(False)

    sh = batch.sched.host()
    costs = algorithmic_costs(wl, sh, sh["n_pull"], sh["n_inner_input"] > 0)
    kernels = []
    for name, (launches, ms) in times.items():
        fl, nb = costs.get(name, (0.0, 0.0))
        per_step_ms = ms / args.steps
        k = {"name": name, "launches_per_step": launches / args.steps,
             "ms_per_step": round(per_step_ms, 4)}
        if fl > 0:
            k["tflops"] = round(fl / (per_step_ms * 1e-3) / 1e12, 2)
        if nb > 0:
            k["gbs"] = round(nb / (per_step_ms * 1e-3) / 1e9, 1)
        kernels.append(k)
    kernels.sort(key=lambda k: -k["ms_per_step"])
    dom = next(k for k in kernels if costs.get(k["name"], (0, 0)) != (0, 0))
    fl, nb = costs[dom["name"]]
    launches, ms = times[dom["name"]]
    avg_ms = ms / launches
    per_launch = fl / (launches / args.steps) if fl > 0 else nb / (launches / args.steps)
    if fl > 0:
        achieved = per_launch / (avg_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_FP32_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_FP32_TFLOPS, 4),
                "traffic": None}
    else:
        achieved = per_launch / (avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None}
    roof["kernel"] = dom["name"]
    roof["avg_launch_us"] = round(avg_ms * 1e3, 2)
    roof["algorithmic_per_launch"] = per_launch

    total_flops = sum(f for f, _ in costs.values())
    out = {
        "metric": METRIC,
        "value": wl.V / (wall_ms * 1e-3),
        "unit": "vertices/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "graphs": wl.K, "vertices": wl.V, "levels": sh["T"],
                   "D": wl.D, "H": wl.H, "loss": "softmax CE at every vertex",
                   "seed": args.seed},
        "roofline": roof,
        "gpu_ms_per_step": round(gpu_ms, 4),
        "schedule_ms": round(sched_ms, 4),
        "fwd_bwd_ms": round(fwdbwd_ms, 4),
        "fwd_bwd_vertices_per_s": wl.V / (fwdbwd_ms * 1e-3),
        "whole_step_tflops": round(total_flops / (wall_ms * 1e-3) / 1e12, 2),
        "algorithmic_gflop_per_step": round(total_flops / 1e9, 3),
        "kernels": kernels[:10],
    }
    if args.cpu_trees > 0:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_trees)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
