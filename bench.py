#!/usr/bin/env python3
"""Throughput of the GCPSL hot path on one MI355X.

A step is one local round of every cluster: cluster-local sampling and
gather, client forward to the cut, server forward/backward, client backward,
SGD update, plus the fusion of all replicas every F rounds -- the whole path,
on inputs already resident in HBM.  The default workload is the 16-cluster
one: K=256 clients, C=16 label-L1 clusters, B=128 per cluster (2048 examples
per step), bf16 activations/weights with fp32 masters, wide residual server,
fusion every 50 rounds, synthetic CIFAR-10-shaped data.  The 8-cluster (bf16)
and 4-cluster (fp32) workloads and the paper's ResNet-18 model (4 clusters,
epoch-barrier schedule, fp32 and bf16) are measured the same way as
sub-results.

Prints one JSON line.  `value` is examples/s summed over the C clusters
(the examples the clusters that take a round process: under the epoch
schedule a cluster whose rounds are done waits at the barrier),
wall clock over exactly --steps rounds bracketed by device synchronisation;
the window is placed so that it ends right after a fusion, so it always holds
at least its share of fusions (exactly its share when F divides --steps).
A second pass right after it records hipEvents around every kernel launch
(on the stream the kernels run on) for per-kernel time; `roofline` gives the
dominant kernel's algorithmic work over that time against the MI355X peak,
and next to it the same fraction from the committed rocprofv3 kernel trace
(profiles/profile.json) with the MFMA busy counters, when the kernel's source
is unchanged since they were taken; `step_roofline` puts the whole step
against the roofline (every kernel's algorithmic work at the peak that bounds
it, over the measured time per step).  The CPU oracle is timed on a bounded
sample on the host cores.
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
    "resnet18": "GCPSL C=4 label-aware (Eq. 4) clusters of K=256 clients, B=64/cluster, fp32, ResNet-18 split "
                "after stage 2 (group norm client / batch norm server), Nesterov SGD with weight decay and "
                "label smoothing, epoch-barrier schedule with fusion after every epoch, synthetic 32x32x3 "
                "10-class",
    "resnet18_bf16": "the same ResNet-18 workload in bf16 (fp32 masters)",
}


def profile(workload, kernel, kind):
    """Figures of the committed rocprofv3 summaries, or None (absent, or the
    kernel's source changed since)."""
    from paper_2609_29395_amd.profile_summary import profile_entry
    return profile_entry(workload, kernel, kind)


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
    us = v["ms"] * 1e3 / v["launches"]
    examples = F * cfg["C"] * cfg["B"]
    # the gather's own work: each example's image read (fp32) and written
    # once in the compute precision, its id and label (4 B each); what the
    # kernel writes beyond that is staging for the first conv layer
    px = cfg["H"] * cfg["W"] * cfg["Cin"]
    alg = examples * (4.0 * px + (2.0 if cfg["dtype"] == "bf16" else 4.0) * px + 8.0)
    impl = v["bytes"] / v["launches"]
    out["gather_window"] = {"kernel": name, "steps": F, "examples": examples, "us": round(us, 1),
                            "algorithmic_bytes": alg, "gbs": round(alg / (us * 1e-6) / 1e9, 1),
                            "frac": round(alg / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
                            "implementation_bytes": impl, "implementation_gbs": round(impl / (us * 1e-6) / 1e9, 1),
                            "implementation_frac": round(impl / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
    del ctxw
    torch.cuda.empty_cache()
    return out


def fusion_aligned_start(warmup, steps, F):
    """First step index >= warmup of a window of `steps` rounds that ends
    right after a fusion (the sampler is stateless in the step index)."""
    if not F:
        return warmup
    return warmup + (-(warmup + steps)) % F


def measure(name, steps, warmup, timing_steps, cpu_seconds, with_cpu=True, with_extras=False, args=None):
    import torch
    from gcpsl_inputs import get_config
    from paper_2609_29395_amd import driver

    cfg = get_config(name)
    C, B = cfg["C"], cfg["B"]
    # the participation table records steps below max_steps; the epoch
    # schedule's fusion interval (slots per epoch) is only known once the
    # context has the assignment, so the table is sized with room for it
    extra = 2 * args.control_steps if with_extras else 0
    ctx, assignment = driver.setup(cfg, max_steps=warmup + steps + timing_steps + extra + 4096)
    if ctx.schedule == "epoch":
        rounds, F = ctx.epoch_rounds()
    else:
        rounds, F = None, cfg["F"]
    x0 = fusion_aligned_start(warmup, steps, F)
    print(f"bench: workload {name} C={C} B={B} F={F} ({ctx.schedule}) warmup={warmup} steps={steps} (timed "
          f"rounds [{x0}, {x0 + steps}))", file=sys.stderr, flush=True)
    driver.train(ctx, warmup, start=x0 - warmup)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    driver.train(ctx, steps, start=x0)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    fusions = (x0 + steps) // F - x0 // F if F else 0
    if rounds is None:
        examples = C * B * steps
    else:  # a cluster whose rounds of the epoch are done waits at the barrier
        examples = B * sum(int((rounds > s % F).sum()) for s in range(x0, x0 + steps))
    value = examples / dt
    print(f"bench: timed {steps} steps ({fusions} fusions, {examples} examples) in {dt:.3f} s", file=sys.stderr,
          flush=True)

    # per-kernel event timing pass, right after the timed window
    ctx.timing(True)
    driver.train(ctx, timing_steps, start=x0 + steps)
    ctx.fuse()  # one fusion inside the per-kernel record
    stats = ctx.timing_read()
    ctx.timing(False)
    dom = max(stats, key=lambda k: stats[k]["ms"])
    st = stats[dom]
    peak_tf = PEAK_TFLOPS[cfg["dtype"]]
    ridge = peak_tf * 1e12 / (PEAK_HBM_GBS * 1e9)
    per_launch_flops = st["flops"] / st["launches"]
    per_launch_bytes = st["bytes"] / st["launches"]
    avg_us = st["ms"] * 1e3 / st["launches"]
    mfma_bound = st["flops"] > 0 and st["flops"] / max(st["bytes"], 1.0) >= ridge
    if mfma_bound:
        achieved = per_launch_flops / (avg_us * 1e-6) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak_tf, "unit": "TFLOP/s",
                "frac": round(achieved / peak_tf, 4)}
    else:
        achieved = per_launch_bytes / (avg_us * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4)}
    tr = profile(name, dom, "traffic")
    roof["traffic"] = None if tr is None else round(tr["bytes_per_launch"], 0)
    roof["kernel"] = dom
    roof["launches"] = st["launches"]
    roof["avg_launch_us"] = round(avg_us, 2)
    roof["work_per_launch"] = per_launch_flops if mfma_bound else per_launch_bytes
    roof["timing"] = (f"hipEvent pair around every launch on the library's stream, {timing_steps} steps run "
                      f"right after the timed window")
    prof_t, prof_m = profile(name, dom, "trace"), profile(name, dom, "mfma")
    if prof_t is not None:
        # the profiled run's launches after its warm-up steps (the steady
        # state this run times), else every launch
        steady = prof_t.get("avg_us_steady")
        prof_us = steady if steady else prof_t["avg_us"]
        rate = roof["work_per_launch"] / (prof_us * 1e-6) / (1e12 if mfma_bound else 1e9)
        roof["profile"] = {"avg_launch_us": round(prof_us, 2), "achieved": round(rate, 2),
                           "frac": round(rate / roof["peak"], 4),
                           "launches": "after the profiled run's warm-up steps" if steady else "every launch",
                           "avg_launch_us_every_launch": round(prof_t["avg_us"], 2),
                           "mfma_busy_pct": None if prof_m is None else round(prof_m["mfma_busy_pct"], 2),
                           "counted_mfma_flops_per_launch": None if prof_m is None else
                           prof_m["counted_flops_per_launch"],
                           "source": f"profiles/profile.json [{name}] (rocprofv3 kernel trace and counters)"}
    else:
        roof["profile"] = None
    conv = {k: v for k, v in stats.items() if k.startswith("conv_")}
    conv_ms = sum(v["ms"] for v in conv.values())
    conv_tf = sum(v["flops"] for v in conv.values()) / (conv_ms * 1e-3) / 1e12 if conv_ms else 0.0
    # MFMA busy of the conv kernels from the counters, weighted by their time
    busy = [(profile(name, k, "mfma"), v["ms"]) for k, v in conv.items()]
    mfma_util = (round(sum(b["mfma_busy_pct"] * ms for b, ms in busy) / sum(ms for _, ms in busy), 2)
                 if busy and all(b is not None for b, _ in busy) else None)
    fuse = stats.get("fuse")
    fusion_gbs = fuse["bytes"] / (fuse["ms"] * 1e-3) / 1e9 if fuse else None
    # the whole step against the roofline: every kernel's algorithmic work at
    # the peak that bounds it (MFMA FLOPs or HBM bytes, whichever takes
    # longer), per step (the fusion at its share of the timed window), over
    # the measured wall time per step
    def ideal_ms(v):
        return 1e3 * max(v["flops"] / (peak_tf * 1e12), v["bytes"] / (PEAK_HBM_GBS * 1e9))
    ideal = sum(ideal_ms(v) for k, v in stats.items() if k != "fuse") / timing_steps
    if fuse:
        ideal += ideal_ms(fuse) / fuse["launches"] * fusions / steps
    step_roof = {"ideal_ms_per_step": round(ideal, 4), "frac": round(ideal / (dt * 1e3 / steps), 4),
                 "definition": "sum over kernels of max(algorithmic FLOPs / MFMA peak, algorithmic bytes / HBM "
                               "peak) per step, over the measured wall time per step"}
    kernel_ms = sum(v["ms"] for v in stats.values())
    for k, v in sorted(stats.items(), key=lambda kv: -kv[1]["ms"]):
        rate = f"{v['flops'] / (v['ms'] * 1e-3) / 1e12:8.1f} TFLOP/s" if v["flops"] > 0 else ""
        print(f"  {k:34s} {v['launches']:5d} launches {v['ms'] / timing_steps:8.3f} ms/step "
              f"{v['bytes'] / (v['ms'] * 1e-3) / 1e9:8.1f} GB/s {rate}", file=sys.stderr)
    out = {
        "value": round(value, 1), "ms_per_step": round(dt * 1e3 / steps, 4), "fusions_in_window": fusions,
        "examples_in_window": examples,
        "dtype": cfg["dtype"],
        "config": {"workload": name, "description": DESCRIPTIONS[name], "clients": cfg["K"], "clusters": C,
                   "batch_per_cluster": B, "global_batch": C * B, "fusion_every": F, "schedule": ctx.schedule,
                   "rule": cfg["rule"],
                   "parallelism": "C replicas batched in every kernel, 1 GPU"},
        "mfma_util_pct": mfma_util,
        "conv_flops_frac_pct": round(100.0 * conv_tf / peak_tf, 2),
        "conv_tflops": round(conv_tf, 2),
        "fusion_gbs": None if fusion_gbs is None else round(fusion_gbs, 1),
        "kernel_ms_per_step": round(kernel_ms / timing_steps, 4),
        "step_roofline": step_roof,
        "roofline": roof,
    }
    if with_extras and not args.no_schedule_control:
        out["schedule_control"] = schedule_control(cfg, ctx, x0 + steps + timing_steps, args.control_steps)
        print(f"bench: schedule control {out['schedule_control']}", file=sys.stderr, flush=True)
    if with_extras and not args.no_hbm_probes:
        out["hbm"] = hbm_probes(cfg, max(F, 1), ctx.cluster_sizes())
        if fusion_gbs is not None:
            out["hbm"]["fusion_in_step"] = {"gbs": round(fusion_gbs, 1),
                                            "frac": round(fusion_gbs / PEAK_HBM_GBS, 4)}
        print(f"bench: hbm {out['hbm']}", file=sys.stderr, flush=True)
    ctx.close()
    del ctx
    torch.cuda.empty_cache()
    if with_cpu:
        out["cpu_baseline"] = cpu_baseline(cfg, assignment, cpu_seconds)
        print(f"bench: cpu baseline {out['cpu_baseline']}", file=sys.stderr, flush=True)
    return out


SUB_RESULTS = ("gcpsl8", "gcpsl4", "resnet18", "resnet18_bf16")


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
    ap.add_argument("--no-sub-results", action="store_true",
                    help="measure only --workload (not also the 8- and 4-cluster and ResNet-18 workloads)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only (--gpus {args.gpus}, WORLD_SIZE {world}); the library "
              "drives one GPU and does not shard the replicas across GPUs", file=sys.stderr)
        sys.exit(2)

    import torch
    torch.cuda.set_device(0)
    head = measure(args.workload, args.steps, args.warmup, args.timing_steps, args.cpu_seconds,
                   with_cpu=not args.no_cpu_baseline, with_extras=True, args=args)
    out = {
        "metric": "examples/s summed over C clusters on 1 GPU; MFMA util %; fusion GB/s",
        "value": head.pop("value"),
        "unit": "examples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head.pop("ms_per_step"),
        "higher_is_better": True,
        "scaling": "strong",
        "vs_baseline": None,
        "dtype": head.pop("dtype"),
        "data": "synthetic",
        "config": head.pop("config"),
    }
    out.update(head)
    if not args.no_sub_results:
        out["sub_results"] = {}
        for name in SUB_RESULTS:
            if name == args.workload:
                continue
            r = measure(name, args.steps, args.warmup, args.timing_steps, args.cpu_seconds / 2,
                        with_cpu=not args.no_cpu_baseline, args=args)
            out["sub_results"][name] = r
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
