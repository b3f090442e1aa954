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

--workload selects one of the other benchmark-shaped batches (tiny, varlstm,
treefc, deep_bf16) for the same report; the default is the headline one.
"""
import argparse
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "Tree-LSTM fwd+bwd vertices/sec (h=512, batch 256); % MFMA / HBM roofline"
PEAK_FP32_TFLOPS = 157.3     # MI355X dense fp32 matrix
PEAK_BF16_TFLOPS = 2500.0    # MI355X dense bf16 matrix
PEAK_HBM_GBS = 8000.0        # MI355X HBM3E


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--workload", default="sst",
                    choices=["sst", "tiny", "varlstm", "treefc", "deep_bf16"])
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU-oracle baseline")
    ap.add_argument("--no-ablation", action="store_true",
                    help="skip the engine ablations (the persistent variant launches "
                         "cooperatively) and the inference passes")
    return ap.parse_args()


def launch_cost(wl, nc, name, row0, rows, n_pull, with_f):
    """Algorithmic (FLOPs, bytes) of one launch.  Level kernels are costed
    over the rows [row0, row0 + rows) they covered; only work the method must
    do counts (absent children and unused gate blocks contribute nothing).
    The lazy and pull products run once per step over all vertices."""
    import numpy as np
    H, D, N = wl.H, wl.D, wl.N
    c = nc[row0:row0 + rows]
    gates_x = 4 if with_f else 3
    if name.startswith(("k_lstm_fwd_level", "k_lstm_bwd_level", "k_lstm_fwd_persist",
                        "k_lstm_bwd_persist", "k_lstm_fwd_tile", "k_lstm_bwd_tile",
                        "k_lstm_fwd_xcd", "k_lstm_bwd_xcd")):
        return float(np.sum(2.0 * H * (3 * H + c * H))), 0.0
    if name.startswith(("k_fc_fwd_tile", "k_fc_bwd_tile", "k_fc_fwd_sk", "k_fc_bwd_sk")):
        return float(np.sum(2.0 * c * H * H)), 0.0
    if name == "k_fc_leaf":            # reads x, writes h and h_out
        return 0.0, rows * H * 4.0 * 3
    if name == "k_lstm_leaf":          # reads 3 columns of P, writes h, c, 5 gates, h_out, c_out
        return 0.0, rows * H * 4.0 * 12
    if name.startswith("k_lstm_bwd_gates"):  # reads dh, dc, 3 gates, c (+ f_k, c_k per child),
        return 0.0, float(np.sum(H * 4.0 * (6 + (3 + N) + 3 * c)))  # writes dA (+ dc_k)
    inner = nc > 0
    lazy = {
        "k_pull_gemm": 2.0 * n_pull * D * gates_x * H,
        "k_pull_leaf<3>": 2.0 * n_pull * D * gates_x * H,
        "k_pull_leaf<4>": 2.0 * n_pull * D * gates_x * H,
        "k_dx_gemm": 2.0 * n_pull * D * gates_x * H,
        "k_dx_tile<64, 64, 3>": 2.0 * n_pull * D * gates_x * H,
        "k_tn_gemm<LdDWx>": 2.0 * n_pull * D * gates_x * H,
        "k_tn_gemm<LdDUiou>": 2.0 * H * (3 if N == 2 else 4) * H * int(inner.sum()),
        "k_tn_gemm<LdDUf>": 2.0 * H * H * float(nc.sum()),
        # one launch per child slot: each carries its share of the links
        "k_tn_gemm<LdFCdW>": 2.0 * H * H * float(nc.sum()) / N,
    }
    if name.startswith("k_tn_group<dUf, dWx"):   # dU_f and dW_x in one grid
        return lazy["k_tn_gemm<LdDUf>"] + lazy["k_tn_gemm<LdDWx>"], 0.0
    if name == "k_tn_group<FCdW>":                  # both child slots in one grid
        return 2.0 * H * H * float(nc.sum()), 0.0
    if name.startswith(("k_dx_tile", "k_pull_tile")):
        return 2.0 * n_pull * D * gates_x * H, 0.0
    base = re.sub(r", (64|128)(, [48])?>", ">", name.replace("_bf", ""))
    base = re.sub(r"^k_tn_dl<(\w+), .*>$", r"k_tn_gemm<\1>", base)
    base = re.sub(r"^k_nt<(\w+)>$", r"k_tn_gemm<\1>", base)   # k_nt_bf, "_bf" dropped
    if name.startswith("k_pack_bf<"):   # bf16 operand packs: fp32 reads, bf16 writes
        MI, nL = int(inner.sum()), float(nc.sum())
        No = 3 * H if N == 2 else 4 * H
        pad = lambda q, m: -(-q // m) * m
        pk = {"LdDUiou": (nL * H + MI * No) * 4.0 + (pad(H, 128) + No) * pad(MI, 64) * 2.0,
              "LdDUf": (nL + 2 * MI) * H * 4.0 + (pad(H, 128) + H) * pad(2 * MI, 64) * 2.0,
              "LdDWx": n_pull * (D + gates_x * H) * 4.0
              + (pad(D, 128) + gates_x * H) * pad(n_pull, 64) * 2.0}
        return 0.0, pk.get(name[len("k_pack_bf<"):-1], 0.0)
    return lazy.get(base, 0.0), 0.0


def source_sha256():
    """Hash of the HIP sources and headers, in the order the traffic record
    was hashed: a record taken on other kernels is not used."""
    import glob
    import hashlib
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(ROOT, "paper_1712_04048_amd", "csrc", "*.hip")) +
                   glob.glob(os.path.join(ROOT, "paper_1712_04048_amd", "csrc", "*.h")) +
                   glob.glob(os.path.join(ROOT, "include", "*.h")))
    for f in sorted(files, key=lambda f: os.path.relpath(f, ROOT)):
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    record (FETCH_SIZE and WRITE_SIZE per dispatch, each scaled by what the
    counter reads for a plain copy of known size), or None when there is no
    record for this kernel or the sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", "traffic_%s.json" % workload)
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    k = rec.get("kernels", {}).get(kernel)
    if k is None or rec.get("source_sha256") != source_sha256():
        return None
    return (k["fetch_kib"] * rec["copy_bytes"] / rec["copy_fetch_kib"] +
            k["write_kib"] * rec["copy_bytes"] / rec["copy_write_kib"])


# graphs in the CPU-oracle samples: (one thread, all cores), chosen so the
# baseline costs about 10-30 s of CPU time on the host next to the GPU
CPU_SAMPLE = {"sst": (48, 256), "tiny": (8, 8), "varlstm": (12, 64), "treefc": (12, 64),
              "deep_bf16": (2, 24)}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def measure_achievable(torch):
    """Rates this device reaches outside the path, as context for the
    roofline: a 1 GiB device-to-device copy (GB/s, read + write) and an
    8192^3 fp32 GEMM through torch's library (TFLOP/s); best of 5 each."""
    out = {}
    a = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1.0)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    best = None
    for _ in range(6):
        e0.record()
        b.copy_(a)
        e1.record()
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1)
        best = t if best is None else min(best, t)
    out["copy_gbs"] = round(2 * a.numel() * 4 / (best * 1e-3) / 1e9, 1)
    del a, b
    n = 8192
    x = torch.randn(n, n, device="cuda")
    y = torch.randn(n, n, device="cuda")
    torch.backends.cuda.matmul.allow_tf32 = False
    best = None
    for _ in range(6):
        e0.record()
        z = x @ y
        e1.record()
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1)
        best = t if best is None else min(best, t)
    out["fp32_gemm_tflops"] = round(2.0 * n ** 3 / (best * 1e-3) / 1e12, 1)
    del x, y, z
    torch.cuda.empty_cache()
    return out


def cpu_baseline(wl, key):
    """The oracle as it stands, in its fp32 build (the same definitions the
    GPU path computes, in the GPU path's precision; bf16 workloads emulate
    the rounding), forward + loss + backward: on one thread over the first
    graphs of the batch, and on all cores (one worker process per core, up
    to 16, each running the oracle on a shard of graphs; partial gradients
    summed in a fixed order) over a larger sample."""
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import oracle
    from parity import OraclePool, subset
    n1, nall = CPU_SAMPLE[key]
    n1, nall = min(n1, wl.K), min(nall, wl.K)
    oracle.lib("f32")
    sub1 = subset(wl, list(range(n1)))
    t0 = time.perf_counter()
    oracle.run(sub1, precision="f32")
    dt1 = time.perf_counter() - t0
    suball = subset(wl, list(range(nall)))
    with OraclePool() as pool:
        pool.run(subset(wl, [0]), precision="f32", backward=False)   # workers started
        t0 = time.perf_counter()
        pool.run(suball, precision="f32")
        dta = time.perf_counter() - t0
        workers = pool.workers
    return {"value": suball.V / dta, "unit": "vertices/s", "cores": workers, "kind": "oracle",
            "sample": "first %d of %d graphs (%d of %d vertices), fp32 build of the recursive "
                      "oracle, forward + loss + backward, %d worker processes (one thread "
                      "each), %.2f s" % (nall, wl.K, suball.V, wl.V, workers, dta),
            "single_thread": {"value": sub1.V / dt1, "unit": "vertices/s", "cores": 1,
                              "sample": "first %d graphs (%d vertices), %.2f s"
                                        % (n1, sub1.V, dt1)},
            "nproc": os.cpu_count(), "cpu_model": cpu_model()}


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
    wl = W.WORKLOADS[args.workload](args.seed)
    lstm = wl.cell == W.CELL_TREE_LSTM
    ctx = B.Context(0)
    batch = Batch(wl, ctx)
    batch.schedule()
    batch.alloc()
    stream = torch.cuda.current_stream()

    for _ in range(args.warmup):
        batch.step()
    ctx.sync()

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
    # per-pass distribution of forward + backward (an event pair per pass)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(max(args.steps, 1))]
    for a, b in evs:
        a.record(stream)
        batch.forward()
        batch.backward()
        b.record(stream)
    torch.cuda.synchronize()
    per_pass = np.array([a.elapsed_time(b) for a, b in evs])
    fwdbwd_pct = {q: round(float(np.percentile(per_pass, q)), 4) for q in (10, 50, 90)}

    # engine ablations (fwd+bwd per pass, HIP events): dU formed level by
    # level instead of lazily, the persistent loop for the small levels, and
    # the backward's children's gates unfused from the level products
    def fwd_bwd_with(*settings):
        # each setting is NAME (set to 1) or NAME=VALUE
        variables = []
        for st in settings:
            var, _, val = st.partition("=")
            os.environ[var] = val or "1"
            variables.append(var)
        try:
            if "CAVS_GENERIC" in variables:   # the generic engine's larger workspace
                batch.alloc()
            batch.forward()
            batch.backward()
            ctx.sync()
            e0.record(stream)
            for _ in range(args.steps):
                batch.forward()
                batch.backward()
            e1.record(stream)
            ctx.sync()
            return e0.elapsed_time(e1) / args.steps
        finally:
            for var in variables:
                del os.environ[var]

    def graph_replay():
        """forward + backward captured once into a HIP graph (through torch's
        stream capture of the library's launches on a side stream), then
        replayed; returns (ms per replay, ms to capture and instantiate)."""
        side = torch.cuda.Stream()
        ctx.set_stream(side)
        try:
            with torch.cuda.stream(side):
                batch.forward()
                batch.backward()
            ctx.sync()
            g = torch.cuda.CUDAGraph()
            tc = time.perf_counter()
            with torch.cuda.graph(g, stream=side):
                batch.forward()
                batch.backward()
            torch.cuda.synchronize()
            cap_ms = (time.perf_counter() - tc) * 1e3
            with torch.cuda.stream(side):
                g.replay()
                e0.record(side)
                for _ in range(args.steps):
                    g.replay()
                e1.record(side)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / args.steps
            del g
            return ms, cap_ms
        finally:
            ctx.set_stream(stream)

    ablation = None
    if lstm and not args.no_ablation:
        ablation = {"unit": "ms per forward + backward pass",
                    "default_engine": round(fwdbwd_ms, 4)}
        ablation["eager_dw_per_level"] = round(fwd_bwd_with("CAVS_EAGER_DW"), 4)
        ablation["persistent_small_levels"] = round(fwd_bwd_with("CAVS_PERSIST",
                                                                 "CAVS_XCD_LOOP=0"), 4)
        ablation["unfused_backward_gates"] = round(fwd_bwd_with("CAVS_UNFUSED_BWD_GATES"), 4)
        ablation["unfused_forward_gates"] = round(fwd_bwd_with("CAVS_UNFUSED_FWD_GATES"), 4)
        ablation["two_stream_lazy_products"] = round(fwd_bwd_with("CAVS_TWO_STREAM"), 4)
        ablation["xcd_loop_off"] = round(fwd_bwd_with("CAVS_XCD_LOOP=0"), 4)
        ablation["xcd_loop_on"] = round(fwd_bwd_with("CAVS_XCD_LOOP=1"), 4)
        ablation["unfused_gates_both"] = round(
            fwd_bwd_with("CAVS_UNFUSED_FWD_GATES", "CAVS_UNFUSED_BWD_GATES"), 4)
        if wl.prec == W.PREC_FP32:
            ablation["generic_engine"] = round(fwd_bwd_with("CAVS_GENERIC"), 4)
        g_ms, cap_ms = graph_replay()
        ablation["graph_captured_replay"] = round(g_ms, 4)
        ablation["graph_capture_instantiate_ms"] = round(cap_ms, 3)

    # inference (cavs_infer: the forward keeping nothing for a backward) beside
    # the training forward alone; whole inference steps include the schedule
    inference = None
    if not args.no_ablation:
        batch.infer()
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(args.steps):
            batch.forward()
        e1.record(stream)
        torch.cuda.synchronize()
        fwd_ms = e0.elapsed_time(e1) / args.steps
        e0.record(stream)
        for _ in range(args.steps):
            batch.infer()
        e1.record(stream)
        torch.cuda.synchronize()
        infer_ms = e0.elapsed_time(e1) / args.steps
        t3 = time.perf_counter()
        for _ in range(args.steps):
            batch.schedule()
            batch.infer()
        torch.cuda.synchronize()
        infer_step_ms = (time.perf_counter() - t3) * 1e3 / args.steps
        inference = {"value": wl.V / (infer_step_ms * 1e-3), "unit": "vertices/s",
                     "step": "cavs_schedule + cavs_infer", "ms_per_step": round(infer_step_ms, 4),
                     "infer_ms": round(infer_ms, 4), "train_forward_ms": round(fwd_ms, 4),
                     "workspace_mb": round(batch.ws_infer.numel() / 2 ** 20, 1),
                     "train_workspace_mb": round(batch.ws.numel() / 2 ** 20, 1)}

    # per-kernel durations: the same steps again with per-launch HIP events
    ctx.timing(True)
    for _ in range(args.steps):
        batch.step()
    recs = ctx.timing_read()
    ctx.timing(False)

    sh = batch.sched.host()
    nc = (sh["child_pos"] >= 0).sum(axis=1)
    with_f = sh["n_inner_input"] > 0
    agg = {}
    for name, row0, rows, ms in recs:
        fl, nb = launch_cost(wl, nc, name, row0, rows, sh["n_pull"], with_f)
        a = agg.setdefault(name, [0, 0.0, 0.0, 0.0])
        a[0] += 1
        a[1] += ms
        a[2] += fl
        a[3] += nb
    # per-level breakdown (microseconds per step) of the level kernels
    per_level = {}
    for name, row0, rows, ms in recs:
        if rows <= 0:
            continue
        kind = ("fwd" if ("fwd" in name or "leaf" in name) else
                "bwd_gates" if "bwd_gates" in name else "bwd_gemm")
        e = per_level.setdefault(row0, {"rows": rows, "fwd": 0.0, "bwd_gates": 0.0,
                                        "bwd_gemm": 0.0})
        e[kind] += ms * 1e3 / args.steps
    level_table = [[v["rows"], round(v["fwd"], 1), round(v["bwd_gates"], 1),
                    round(v["bwd_gemm"], 1)] for _, v in sorted(per_level.items())]
    kernels = []
    for name, (launches, ms, fl, nb) in agg.items():
        k = {"name": name, "launches_per_step": launches / args.steps,
             "ms_per_step": round(ms / args.steps, 4)}
        if fl > 0:
            k["tflops"] = round(fl / (ms * 1e-3) / 1e12, 2)
        if nb > 0:
            k["gbs"] = round(nb / (ms * 1e-3) / 1e9, 1)
        kernels.append(k)
    kernels.sort(key=lambda k: -k["ms_per_step"])
    dom = next(k for k in kernels if agg[k["name"]][2] > 0 or agg[k["name"]][3] > 0)
    launches, ms, fl, nb = agg[dom["name"]]
    avg_ms = ms / launches
    if fl > 0:
        per_launch = fl / launches
        achieved = per_launch / (avg_ms * 1e-3) / 1e12
        bf = "_bf" in dom["name"] or ", true>" in dom["name"] or ", true," in dom["name"]
        peak = PEAK_BF16_TFLOPS if bf else PEAK_FP32_TFLOPS
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak,
                "unit": "TFLOP/s", "frac": round(achieved / peak, 4), "traffic": None}
    else:
        per_launch = nb / launches
        achieved = per_launch / (avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None}
    roof["traffic"] = measured_traffic(wl.name, dom["name"])
    if roof["traffic"] is not None:
        roof["traffic"] = round(roof["traffic"])
        roof["traffic_unit"] = "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)"
    roof["kernel"] = dom["name"]
    roof["launches_per_step"] = launches / args.steps
    roof["avg_launch_us"] = round(avg_ms * 1e3, 2)
    roof["algorithmic_per_launch"] = per_launch

    total_flops = sum(a[2] for a in agg.values()) / args.steps
    # the whole step against the matrix peak of its precision (every
    # workload here is bound by its products at the roofline), and the
    # achievable rates measured on this device for context: a plain device
    # copy and a large library fp32 GEMM (torch), neither part of the path
    step_peak = PEAK_BF16_TFLOPS if wl.prec == W.PREC_BF16 else PEAK_FP32_TFLOPS
    t_roof_us = total_flops / (step_peak * 1e12) * 1e6
    achievable = measure_achievable(torch)
    if roof["unit"] == "TFLOP/s" and roof["peak"] == PEAK_FP32_TFLOPS:
        roof["frac_of_library_fp32_gemm"] = round(roof["achieved"] /
                                                  achievable["fp32_gemm_tflops"], 4)
    elif roof["unit"] == "GB/s":
        roof["frac_of_copy"] = round(roof["achieved"] / achievable["copy_gbs"], 4)
    loss_desc = ("softmax CE at every vertex" if wl.loss == W.LOSS_CE and
                 (wl.push_idx >= 0).all() else
                 "softmax CE at the roots" if wl.loss == W.LOSS_CE else "L2 at the roots")
    out = {
        "metric": METRIC if args.workload == "sst" else
        "%s fwd+bwd vertices/sec" % wl.name,
        "value": wl.V / (wall_ms * 1e-3),
        "unit": "vertices/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.prec == W.PREC_BF16 else "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "graphs": wl.K, "vertices": wl.V, "levels": sh["T"],
                   "D": wl.D, "H": wl.H, "loss": loss_desc, "seed": args.seed},
        "roofline": roof,
        "gpu_ms_per_step": round(gpu_ms, 4),
        "schedule_ms": round(sched_ms, 4),
        "fwd_bwd_ms": round(fwdbwd_ms, 4),
        "fwd_bwd_vertices_per_s": wl.V / (fwdbwd_ms * 1e-3),
        "whole_step_tflops": round(total_flops / (wall_ms * 1e-3) / 1e12, 2),
        "whole_step_roofline": {"bound": "mfma", "peak_tflops": step_peak,
                                "t_roof_us": round(t_roof_us, 1),
                                "frac": round(t_roof_us * 1e-3 / wall_ms, 4)},
        "fwd_bwd_ms_p10_p50_p90": [fwdbwd_pct[10], fwdbwd_pct[50], fwdbwd_pct[90]],
        "achievable": achievable,
        "algorithmic_gflop_per_step": round(total_flops / 1e9, 3),
        "kernels": kernels,
        "levels_us": {"columns": ["rows", "fwd", "bwd_gates", "bwd_gemm"], "rows": level_table},
    }
    if ablation is not None:
        out["ablation"] = ablation
    if inference is not None:
        out["inference"] = inference
    ctx.sync()
    batch = None
    ctx.close()
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(wl, args.workload)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
