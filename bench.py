#!/usr/bin/env python3
"""Throughput of the GCPSL hot path on one MI355X.

A step is one local round of every cluster: cluster-local sampling and
gather, client forward to the cut, server forward/backward, client backward,
SGD update, plus the fusion of all replicas every F rounds -- the whole path,
on inputs already resident in HBM.  The default workload is the 16-cluster
one: K=256 clients, C=16 label-L1 clusters, B=128 per cluster (2048 examples
per step), bf16 activations/weights with fp32 masters, wide residual server,
fusion every 50 rounds, synthetic CIFAR-10-shaped data.

Prints one JSON line.  `value` is examples/s summed over the C clusters,
wall clock over exactly --steps rounds bracketed by device synchronisation.
A second, separately timed pass records hipEvents around every kernel launch
(on the stream the kernels run on) to report the dominant kernel's roofline
fraction.  The CPU oracle is timed on a bounded sample on the host cores.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# MI355X published peaks
PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
PEAK_HBM_GBS = 8000.0

DESCRIPTIONS = {
    "gcpsl16": "GCPSL C=16 label-L1 clusters of K=256 clients, B=128/cluster, bf16 (fp32 masters), "
               "split CNN 3-32-64|64-256-3x256res, fusion every 50 rounds, synthetic 32x32x3 10-class",
    "gcpsl8": "GCPSL C=8 size-balanced clusters of K=256 clients, B=64/cluster, bf16 (fp32 masters), "
              "split CNN 3-32-64|64-128-128, fusion every 25 rounds, synthetic 32x32x3 10-class",
    "gcpsl4": "GCPSL C=4 random clusters of K=256 clients, B=64/cluster, fp32, "
              "split CNN 3-32-64|64-128-128, fusion every 50 rounds, synthetic 32x32x3 10-class",
    "gpsl": "GPSL C=1, K=256 clients, B=64, fp32, split CNN 3-32-64|64-128-128, synthetic 32x32x3",
}


def load_traffic(workload, kernel):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when it is absent or the kernel's source changed since it was taken."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    from paper_2609_29395_amd.profile_summary import file_hash, kernel_source
    with open(path) as fh:
        rec = json.load(fh)
    src = kernel_source(kernel)
    if rec.get("source_hashes", {}).get(src) != file_hash(src):
        return None
    entry = rec.get("kernels", {}).get(f"{workload}:{kernel}")
    return None if entry is None else entry.get("bytes_per_launch")


def cpu_baseline(cfg, assignment, budget_s):
    """Oracle rounds of cluster 0 on the host cores until budget_s elapses."""
    from threadpoolctl import threadpool_info
    from oracle.train import GCPSLOracle
    o = GCPSLOracle(cfg, cluster_of_client=assignment)
    o.round(0, replicas=[0])  # warm the BLAS pools
    t0 = time.perf_counter()
    rounds = 0
    while True:
        o.round(1 + rounds, replicas=[0])
        rounds += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    return {"value": round(cfg["B"] * rounds / dt, 3), "unit": "examples/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{rounds} local rounds of one cluster (B={cfg['B']} examples each: sampling, gather, "
                      f"split forward/backward, SGD) of the {cfg['name']} workload in fp64 numpy, "
                      f"{dt:.1f} s; the rate per example equals the C-cluster rate"}


def _timed(fn):
    import torch
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    fn()
    torch.cuda.synchronize()
    return time.perf_counter() - t0


def schedule_control(cfg, ctx, start, steps):
    """Concurrent against sequential execution of the cluster workloads on
    this GPU (the one-GPU analogue of Eq. 6's comparison): the same rounds,
    once with all clusters of a step in one launch per kernel, once with the
    clusters run one after another through gcpsl_step_replica.  Lockstep:
    `steps` rounds of the workload's own schedule.  Epoch barrier: one system
    epoch of R slots in which cluster n takes r_n = floor(n_n / B) rounds."""
    from paper_2609_29395_amd import driver
    out = {}
    conc = _timed(lambda: driver.train(ctx, steps, start=start))
    seq = _timed(lambda: driver.train(ctx, steps, start=start + steps, serial=True))
    out["lockstep"] = {"rounds_per_cluster": steps, "concurrent_ms_per_step": round(conc * 1e3 / steps, 3),
                       "sequential_ms_per_step": round(seq * 1e3 / steps, 3), "speedup": round(seq / conc, 3)}
    ectx, _ = driver.setup(cfg, max_steps=1, schedule="epoch")
    rounds, R = ectx.epoch_rounds()
    driver.train(ectx, min(R, 4), start=0)  # warm-up slots
    conc = _timed(lambda: driver.train(ectx, R, start=R))
    seq = _timed(lambda: driver.train(ectx, R, start=2 * R, serial=True))
    work = int(rounds.sum())
    out["epoch"] = {"slots_per_epoch": int(R), "cluster_rounds_per_epoch": work,
                    "eq6_ideal_speedup": round(work / R, 3),
                    "concurrent_s": round(conc, 4), "sequential_s": round(seq, 4), "speedup": round(seq / conc, 3),
                    "concurrent_examples_per_s": round(work * cfg["B"] / conc, 1)}
    ectx.close()
    return out


def hbm_probes(cfg, F, ctx_sizes):
    """The HBM-bound kernels at sizes where launch ramps and the 256 MB MALL
    do not decide the rate: the fusion kernel on 16 replicas of 16M + 2
    parameters (2.1 GB read, 2.1 GB written; weights = the workload's cluster
    sizes) through gcpsl_fuse_replicas, and the gather of an F-step sample
    window (gcpsl_sample with nsteps = F).  Rates are algorithmic bytes over
    hipEvent time on the launching stream."""
    import numpy as np
    import torch
    from paper_2609_29395_amd import driver, gcpsl

    out = {}
    Cf, Pf = 16, 16 * 1024 * 1024 + 2
    w = np.resize(np.asarray(ctx_sizes, dtype=np.int64), Cf)
    theta = torch.randn(Cf, Pf, device="cuda", generator=torch.Generator(device="cuda").manual_seed(0))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for _ in range(2):
        gcpsl.fuse_replicas(theta, w)
    reps = 5
    e0.record()
    for _ in range(reps):
        gcpsl.fuse_replicas(theta, w)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / reps
    fb = 8.0 * Cf * Pf
    out["fusion_16x16M"] = {"replicas": Cf, "params": Pf, "bytes": fb, "us": round(us, 1),
                            "gbs": round(fb / (us * 1e-6) / 1e9, 1),
                            "frac": round(fb / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
    del theta
    torch.cuda.empty_cache()

    ctxw, _ = driver.setup(cfg, max_steps=4 * F, max_window=F)
    ctxw.sample(0, F)
    torch.cuda.synchronize()
    ctxw.timing(True)
    for k in range(1, 4):
        ctxw.sample(k * F, F)
    st = ctxw.timing_read()
    ctxw.timing(False)
    g = {k: v for k, v in st.items() if k.startswith("gather")}
    name, v = max(g.items(), key=lambda kv: kv[1]["bytes"])
    gbs = v["bytes"] / (v["ms"] * 1e-3) / 1e9
    out["gather_window"] = {"kernel": name, "steps": F, "examples": F * cfg["C"] * cfg["B"],
                            "bytes": v["bytes"] / v["launches"], "us": round(v["ms"] * 1e3 / v["launches"], 1),
                            "gbs": round(gbs, 1), "frac": round(gbs / PEAK_HBM_GBS, 4)}
    del ctxw
    torch.cuda.empty_cache()
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="gcpsl16", choices=sorted(DESCRIPTIONS))
    ap.add_argument("--timing-steps", type=int, default=20)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-schedule-control", action="store_true",
                    help="skip the concurrent-vs-sequential cluster execution control")
    ap.add_argument("--control-steps", type=int, default=10)
    ap.add_argument("--no-hbm-probes", action="store_true",
                    help="skip the large fusion and windowed gather measurements")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only (--gpus {args.gpus}, WORLD_SIZE {world}); the multi-GPU "
              "fusion path is a design, not part of this build", file=sys.stderr)
        sys.exit(2)

    import torch
    from gcpsl_inputs import get_config
    from paper_2609_29395_amd import driver

    cfg = get_config(args.workload)
    C, B, F = cfg["C"], cfg["B"], cfg["F"]
    total = args.warmup + args.steps + args.timing_steps + 2 * args.control_steps
    print(f"bench: workload {args.workload} C={C} B={B} F={F} warmup={args.warmup} steps={args.steps}",
          file=sys.stderr, flush=True)
    torch.cuda.set_device(0)
    ctx, assignment = driver.setup(cfg, max_steps=total)
    stream = torch.cuda.current_stream()

    driver.train(ctx, args.warmup, start=0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    driver.train(ctx, args.steps, start=args.warmup)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    value = C * B * args.steps / dt
    print(f"bench: timed {args.steps} steps in {dt:.3f} s", file=sys.stderr, flush=True)

    # per-kernel event timing pass (separate from the timed region)
    ctx.timing(True)
    driver.train(ctx, args.timing_steps, start=args.warmup + args.steps)
    ctx.fuse()  # one fusion inside the timed-kernel record
    stats = ctx.timing_read()
    ctx.timing(False)
    nsteps = args.timing_steps
    dom = max(stats, key=lambda k: stats[k]["ms"])
    st = stats[dom]
    ridge = PEAK_TFLOPS[cfg["dtype"]] * 1e12 / (PEAK_HBM_GBS * 1e9)
    intensity = st["flops"] / max(st["bytes"], 1.0)
    if st["flops"] > 0 and intensity >= ridge:
        achieved = st["flops"] / (st["ms"] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_TFLOPS[cfg["dtype"]],
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_TFLOPS[cfg["dtype"]], 4)}
    else:
        achieved = st["bytes"] / (st["ms"] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4)}
    traffic = load_traffic(args.workload, dom)
    roof["traffic"] = traffic
    roof["kernel"] = dom
    roof["launches"] = st["launches"]
    roof["avg_launch_us"] = round(st["ms"] * 1e3 / st["launches"], 2)
    conv = [v for k, v in stats.items() if k.startswith("conv_")]
    conv_ms = sum(v["ms"] for v in conv)
    conv_tf = sum(v["flops"] for v in conv) / (conv_ms * 1e-3) / 1e12 if conv_ms else 0.0
    fuse = stats.get("fuse")
    fusion_gbs = fuse["bytes"] / (fuse["ms"] * 1e-3) / 1e9 if fuse else None
    kernel_ms = sum(v["ms"] for v in stats.values())
    breakdown = sorted(((k, v) for k, v in stats.items()), key=lambda kv: -kv[1]["ms"])
    for k, v in breakdown:
        rate = (f"{v['flops'] / (v['ms'] * 1e-3) / 1e12:8.1f} TFLOP/s" if v["flops"] > 0 else "")
        print(f"  {k:34s} {v['launches']:5d} launches {v['ms'] / nsteps:8.3f} ms/step "
              f"{v['bytes'] / (v['ms'] * 1e-3) / 1e9:8.1f} GB/s {rate}", file=sys.stderr)

    out = {
        "metric": "examples/s summed over C clusters on 1 GPU; MFMA util %; fusion GB/s",
        "value": round(value, 1),
        "unit": "examples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(dt * 1e3 / args.steps, 4),
        "higher_is_better": True,
        "scaling": "strong",
        "vs_baseline": None,
        "dtype": cfg["dtype"],
        "data": "synthetic",
        "config": {"workload": args.workload, "description": DESCRIPTIONS[args.workload], "clients": cfg["K"],
                   "clusters": C, "batch_per_cluster": B, "global_batch": C * B, "fusion_every": F,
                   "rule": cfg["rule"], "parallelism": "C replicas batched in every kernel, 1 GPU"},
        "mfma_util_pct": round(100.0 * conv_tf / PEAK_TFLOPS[cfg["dtype"]], 2),
        "conv_tflops": round(conv_tf, 2),
        "fusion_gbs": None if fusion_gbs is None else round(fusion_gbs, 1),
        "kernel_ms_per_step": round(kernel_ms / nsteps, 4),
        "roofline": roof,
    }
    if not args.no_schedule_control:
        out["schedule_control"] = schedule_control(cfg, ctx, args.warmup + args.steps + args.timing_steps,
                                                   args.control_steps)
        print(f"bench: schedule control {out['schedule_control']}", file=sys.stderr, flush=True)
    if not args.no_hbm_probes:
        out["hbm"] = hbm_probes(cfg, max(F, 1), ctx.cluster_sizes())
        if fusion_gbs is not None:
            out["hbm"]["fusion_in_step"] = {"gbs": round(fusion_gbs, 1), "frac": round(fusion_gbs / PEAK_HBM_GBS, 4)}
        print(f"bench: hbm {out['hbm']}", file=sys.stderr, flush=True)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, assignment, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
