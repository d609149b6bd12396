"""Summaries of rocprofv3 output for the kernels of this library.

Every figure lands in profiles/profile.json, per workload and kernel label,
with the hash of each kernel source file at the time it was taken (bench.py
reports a figure only while the kernel's source still has that hash), and in
a Markdown summary per workload and kind:

  python -m paper_2609_29395_amd.profile_summary copy [--mib N] [--reps R]
      Run a plain device copy of a known size (the calibration kernel for the
      FETCH_SIZE / WRITE_SIZE counters).
  python -m paper_2609_29395_amd.profile_summary stats TRACE_DIR WORKLOAD OUT.md CMD...
      `rocprofv3 --kernel-trace --stats` CSV output: calls, total and average
      duration per kernel.
  python -m paper_2609_29395_amd.profile_summary mfma PMC_DIR WORKLOAD OUT.md CMD...
      `rocprofv3 --pmc SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16
      SQ_INSTS_VALU_MFMA_MOPS_F32 GRBM_GUI_ACTIVE` CSV output: MFMA busy
      fraction (busy cycles over GUI-active cycles times the 1024 SIMDs) and
      MFMA FLOPs counted per launch (512 per MOPS count).
  python -m paper_2609_29395_amd.profile_summary traffic FETCH_DIR WRITE_DIR COPY_FETCH_DIR COPY_WRITE_DIR WORKLOAD OUT.md
      Two counter runs of the workload (FETCH_SIZE, then WRITE_SIZE) combined
      into HBM bytes per launch for every kernel, each counter scaled by what
      it reads for the copy of known size (runs COPY_FETCH_DIR, COPY_WRITE_DIR).
  python -m paper_2609_29395_amd.profile_summary layers TRACE_DIR OUT.md CMD...
      Per-dispatch table of one step from `rocprofv3 --kernel-trace` CSV output.
  python -m paper_2609_29395_amd.profile_summary gemm-ref OUT.md
      hipBLASLt bf16 GEMMs of the convolution shapes, for comparison.
"""
from __future__ import annotations

import collections
import csv
import glob
import hashlib
import json
import os
import re
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
COPY_MIB = 256
PROFILE_JSON = os.path.join(ROOT, "profiles", "profile.json")
SIMDS = 256 * 4  # MI355X: 256 compute units of 4 SIMDs


def kernel_label(name: str) -> str:
    """rocprof's demangled name -> the label gcpsl_timing reports."""
    m = re.search(r"conv_kernel<(unsigned short|float), (\d+), (\d+), (\d+), (\d+), (true|false), (\d), "
                  r"(\d+), (\d+), (\d+)>", name)
    if m:
        t = "bf16" if m.group(1) == "unsigned short" else "f32"
        kind = "conv_fwd" if m.group(7) == "0" else "conv_dgrad"
        w = int(m.group(4)) * int(m.group(5))
        k = int(m.group(9)) // (2 if t == "bf16" else 4)
        return (f"{kind}<{t},{m.group(2)}x{m.group(3)}x{k},w{w},"
                f"{'vec' if m.group(6) == 'true' else 'gather'}>")
    m = re.search(r"wgrad_kernel<(unsigned short|float), (\d+), (\d+), (\d+), (\d+), (true|false)>", name)
    if m:
        t = "bf16" if m.group(1) == "unsigned short" else "f32"
        w = int(m.group(4)) * int(m.group(5))
        return f"conv_wgrad<{t},{m.group(2)}x{m.group(3)},w{w},{'vec' if m.group(6) == 'true' else 'gather'}>"
    # (an optional last flag marks the halo forward that also writes the image means)
    m = re.search(r"conv_lds_kernel<(\d+), (\d+), (\d+), (\d+), (\d), (true|false)(, (true|false))?"
                  r"(, (true|false))?(, (\d))?>", name)
    if m:
        kind = "conv_fwd" if m.group(5) == "0" else "conv_dgrad"
        w = int(m.group(3)) * int(m.group(4))
        mode = "halo" if m.group(8) == "true" else "lds"
        if mode == "halo" and m.group(12) == "1":  # one halo buffer
            return f"{kind}<bf16,{m.group(1)}x{m.group(2)}x64,w{w},halo1>"
        kt = 192 if (mode == "halo" and m.group(2) == "64") else 64  # tap-row k tiles
        return f"{kind}<bf16,{m.group(1)}x{m.group(2)}x{kt},w{w},{mode}>"
    m = re.search(r"conv_img_kernel<(\d+), (\d+), (\d)(, (\d))?>", name)
    if m:  # (a last argument: image rows per wave, 256 pixels per tile each)
        kind = "conv_fwd" if m.group(3) == "0" else "conv_dgrad"
        tile = 256 * int(m.group(5) or 1)
        return f"{kind}<bf16,{tile}x{m.group(2)}x{9 * int(m.group(1))},w8,img>"
    m = re.search(r"conv_img_pool_kernel<(\d+)>", name)
    if m:  # the persistent forward into the max pool and its routing codes
        return f"conv_fwd<bf16,512x{m.group(1)}x288,w8,img,pool>"
    if re.search(r"conv_img_dgrad_kernel\b", name):  # the persistent input gradient from the pooled gradient
        return "conv_dgrad<bf16,256x32x576,w8,img,pool>"
    m = re.search(r"wgrad_col_kernel(<(true|false)>)?", name)
    if m:
        return "conv_wgrad<bf16,32x27,w4,img3>" if m.group(2) == "true" else "conv_wgrad<bf16,32x32,w4,col>"
    m = re.search(r"conv_col_kernel(<(true|false)>)?", name)
    if m:
        return "conv_fwd<bf16,256x32x27,w4,img3>" if m.group(2) == "true" else "conv_fwd<bf16,256x32x32,w4,col>"
    m = re.search(r"wgrad_img_kernel<\d+(, (true|false))?>", name)
    if m:  # (true: the output gradient routed from a max pool's codes)
        return "conv_wgrad<bf16,64x288,w8,img,pool>" if m.group(2) == "true" else "conv_wgrad<bf16,64x288,w8,img>"
    if re.search(r"wgrad_halo_kernel<", name):
        return "conv_wgrad<bf16,128x576,w8,halo>"
    m = re.search(r"wgrad_lds_kernel<(\d+), (\d+), (\d+), (\d+), (?:\d+, \d+, )?(true|false)>", name)
    if m:
        w = int(m.group(3)) * int(m.group(4))
        return f"conv_wgrad<bf16,{m.group(1)}x{m.group(2)},w{w},lds>"
    if re.search(r"sgd_seg_kernel<", name):
        return "sgd"  # the update with the split-K sums, the library's "sgd" launch
    m = re.search(r"::(\w+?)(_kernel)?[<(]", name)
    return m.group(1) if m else name


CSRC = os.path.join(ROOT, "paper_2609_29395_amd", "csrc")
SHARED_HEADERS = ("common.h",)  # device helpers every kernel source includes


def kernel_source(label: str) -> str:
    """The source file that holds the kernel a timing label names."""
    if label.startswith("conv_wgrad<") and label.endswith((",lds>", ",halo>", ",img>", ",col>", ",img3>", ",pool>")):
        return "k_wgrad_lds.hip"
    if label.startswith("conv_") and label.endswith((",lds>", ",halo>", ",halo1>")):
        return "k_conv_lds.hip"
    if label.startswith("conv_") and label.endswith((",img>", ",col>", ",img3>", ",img,pool>")):
        return "k_conv_img.hip"
    if label.startswith("conv_"):
        return "k_conv.hip"
    if label in ("chan_reduce", "chan_finish", "group_reduce", "norm_apply_fwd", "norm_apply_bwd") or \
            label.startswith(("batchnorm", "groupnorm")):
        return "k_norm.hip"
    if label in ("im2col", "zero_insert"):
        return "k_block.hip"
    return "k_misc.hip"


def file_hash(name: str) -> str:
    """Hash of one kernel source together with the shared device headers."""
    h = hashlib.sha256()
    for f in (name, *SHARED_HEADERS):
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def source_hashes() -> dict:
    return {f: file_hash(f) for f in sorted(os.listdir(CSRC)) if f.endswith(".hip")}


def copy(mib=COPY_MIB, reps=5):
    import torch
    n = mib * 1024 * 1024 // 4
    a = torch.ones(n, device="cuda")
    b = torch.empty_like(a)
    for _ in range(reps):
        b.copy_(a)
    torch.cuda.synchronize()
    print(f"copied {mib} MiB x {reps}")


def _one(pattern):
    files = glob.glob(pattern, recursive=True)
    if not files:
        raise FileNotFoundError(pattern)
    return files[0]


def _update_profile(workload, kind, entries):
    """Set the {label: {field: value}} of one kind (trace, mfma, traffic) of a
    workload in profiles/profile.json, with the current source hash of each
    label's file; labels of that kind the new run does not have are dropped."""
    rec = {}
    if os.path.exists(PROFILE_JSON):
        with open(PROFILE_JSON) as fh:
            rec = json.load(fh)
    w = rec.setdefault(workload, {})
    for lab in list(w):
        if lab not in entries:
            w[lab].pop(kind, None)
            if not w[lab]:
                del w[lab]
    for lab, fields in entries.items():
        e = w.setdefault(lab, {})
        e[kind] = dict(fields, source_hash=file_hash(kernel_source(lab)))
    with open(PROFILE_JSON, "w") as fh:
        json.dump(rec, fh, indent=1, sort_keys=True)


def profile_entry(workload, label, kind):
    """One kind of profile figures for a kernel, or None when absent or taken
    on a source file that has changed since."""
    if not os.path.exists(PROFILE_JSON):
        return None
    with open(PROFILE_JSON) as fh:
        rec = json.load(fh)
    e = rec.get(workload, {}).get(label, {}).get(kind)
    if e is None or e.get("source_hash") != file_hash(kernel_source(label)):
        return None
    return e


def steady_averages(trace_dir, warmup):
    """Per label, the mean launch duration (us) over the launches that start
    after the warm-up steps of the bench run: the sampler runs once per step,
    so its (warmup + 1)-th launch starts the first step after the warm-up."""
    try:
        rows = list(csv.DictReader(open(_one(os.path.join(trace_dir, "**", "*kernel_trace.csv")))))
    except FileNotFoundError:
        return {}
    starts = sorted(int(r["Start_Timestamp"]) for r in rows if "sample_kernel" in r["Kernel_Name"])
    t0 = starts[warmup] if 0 < warmup < len(starts) else 0
    by = collections.defaultdict(list)
    for r in rows:
        if int(r["Start_Timestamp"]) >= t0:
            by[kernel_label(r["Kernel_Name"])].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    return {lab: sum(v) / len(v) for lab, v in by.items()}


def stats(trace_dir, workload, out_md, cmd):
    rows = list(csv.DictReader(open(_one(os.path.join(trace_dir, "**", "*kernel_stats.csv")))))
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    # instantiations that share a label (e.g. the head conv that also writes
    # the pooled features) are one row, as in the library's own timing
    by = collections.defaultdict(lambda: [0, 0.0])
    for r in rows:
        v = by[kernel_label(r["Name"])]
        v[0] += int(r["Calls"])
        v[1] += float(r["TotalDurationNs"])
    m = re.search(r"--warmup (\d+)", " ".join(cmd))
    warmup = int(m.group(1)) if m else 0
    steady = steady_averages(trace_dir, warmup)
    lines = [f"# Kernel time summary, {workload}", "", f"Command: `{' '.join(cmd)}`", "",
             f"avg us: every launch of the run (rocprofv3 --stats); after warm-up: the launches of the steps "
             f"after the run's {warmup} warm-up steps (kernel trace), the steady state the bench times.", "",
             "| kernel (label) | calls | total ms | avg us | avg us after warm-up | % |", "|---|---|---|---|---|---|"]
    for lab, (calls, tot) in sorted(by.items(), key=lambda kv: -kv[1][1]):
        st = f"{steady[lab]:.2f}" if lab in steady else "-"
        lines.append(f"| {lab} | {calls} | {tot / 1e6:.3f} | {tot / calls / 1e3:.2f} | {st} | {100 * tot / total:.2f} |")
    lines += ["", f"Sum of kernel time: {total / 1e6:.3f} ms", ""]
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))
    _update_profile(workload, "trace", {lab: {"calls": c, "avg_us": t / c / 1e3, "avg_us_steady": steady.get(lab)}
                                        for lab, (c, t) in by.items()
                                        if not lab.startswith(("elementwise", "vectorized", "__amd"))})


def mfma(pmc_dir, workload, out_md, cmd):
    """MFMA busy fraction and counted MFMA FLOPs per launch, per kernel label."""
    rows = list(csv.DictReader(open(_one(os.path.join(pmc_dir, "**", "*counter_collection.csv")))))
    disp = collections.defaultdict(dict)  # dispatch id -> {counter: value, name, ns}
    for r in rows:
        d = disp[r["Dispatch_Id"]]
        d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        d["name"] = r["Kernel_Name"]
        d["ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    by = collections.defaultdict(list)
    for d in disp.values():
        lab = kernel_label(d["name"])
        if not lab.startswith(("elementwise", "vectorized", "__amd")):
            by[lab].append(d)

    def gui_per_xcd(d):
        g = d.get("GRBM_GUI_ACTIVE", 0.0)
        return g / 8.0 if d["ns"] > 0 and g > 3.0 * d["ns"] else g  # the CSV sums the 8 XCDs

    out = {}
    lines = [f"# MFMA counters per launch, {workload}", "", f"Command: `{' '.join(cmd)}`", "",
             "MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE x 1024 SIMDs), with GRBM_GUI_ACTIVE per "
             "XCD (the CSV value over 8 when it sums the 8 XCDs, i.e. when it exceeds the launch's duration "
             "times 3 GHz); counted FLOPs = 512 x SQ_INSTS_VALU_MFMA_MOPS_{BF16,F32}; GUI-active MHz = "
             "GRBM_GUI_ACTIVE per XCD over the launch's duration.", "",
             "| kernel (label) | launches | MFMA busy % | counted MFMA GFLOP/launch | GUI-active MHz |",
             "|---|---|---|---|---|"]
    for lab, ds in by.items():
        busy = sum(d.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) for d in ds)
        gui = sum(gui_per_xcd(d) for d in ds)
        flops = 512.0 * sum(d.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) + d.get("SQ_INSTS_VALU_MFMA_MOPS_F32", 0.0)
                            for d in ds) / len(ds)
        ns = sum(d["ns"] for d in ds)
        out[lab] = {"launches": len(ds), "mfma_busy_pct": 100.0 * busy / (gui * SIMDS) if gui > 0 else 0.0,
                    "counted_flops_per_launch": flops, "gui_mhz": 1e3 * gui / ns if ns > 0 else 0.0}
    for lab, v in sorted(out.items(), key=lambda kv: -kv[1]["counted_flops_per_launch"]):
        lines.append(f"| {lab} | {v['launches']} | {v['mfma_busy_pct']:.1f} | "
                     f"{v['counted_flops_per_launch'] / 1e9:.2f} | {v['gui_mhz']:.0f} |")
    lines.append("")
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))
    _update_profile(workload, "mfma", out)


def _counter_per_dispatch(d, counter):
    rows = list(csv.DictReader(open(_one(os.path.join(d, "**", "*counter_collection.csv")))))
    per = collections.defaultdict(list)
    for r in rows:
        if r["Counter_Name"] == counter:
            per[r["Kernel_Name"]].append(float(r["Counter_Value"]))
    return per


def traffic(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, workload, out_md):
    fetch = _counter_per_dispatch(fetch_dir, "FETCH_SIZE")
    write = _counter_per_dispatch(write_dir, "WRITE_SIZE")
    expect_kib = COPY_MIB * 1024.0
    samples = lambda per: [v for vs in per.values() for v in vs if v > 0.25 * expect_kib]
    cf = samples(_counter_per_dispatch(copy_fetch_dir, "FETCH_SIZE"))
    cw = samples(_counter_per_dispatch(copy_write_dir, "WRITE_SIZE"))
    f_fac = (sum(cf) / len(cf)) / expect_kib if cf else 1.0
    w_fac = (sum(cw) / len(cw)) / expect_kib if cw else 1.0
    # per label: the launches of every instantiation with that label
    fl, wl = collections.defaultdict(list), collections.defaultdict(list)
    for k, v in fetch.items():
        fl[kernel_label(k)] += v
    for k, v in write.items():
        wl[kernel_label(k)] += v
    out = {}
    for k in set(fl) | set(wl):
        if k.startswith(("elementwise", "vectorized", "__amd")):
            continue
        fv, wv = fl.get(k, []), wl.get(k, [])
        fk = sum(fv) / len(fv) if fv else 0.0
        wk = sum(wv) / len(wv) if wv else 0.0
        out[k] = {"launches": max(len(fv), len(wv)), "fetch_kib": fk, "write_kib": wk,
                  "fetch_factor": f_fac, "write_factor": w_fac,
                  "bytes_per_launch": 1024.0 * (fk / f_fac + wk / w_fac)}
    lines = [f"# HBM traffic per launch, {workload}", "",
             "Commands (R = repository root; O = an output directory; B = the bench.py command of the "
             "kernel-trace summary of this workload):", "",
             "* `rocprofv3 --pmc FETCH_SIZE --output-format csv -d $O/pfetch -o run -- $B`",
             "* `rocprofv3 --pmc WRITE_SIZE --output-format csv -d $O/pwrite -o run -- $B`",
             "* `rocprofv3 --pmc FETCH_SIZE --output-format csv -d $O/cfetch -o run -- python "
             "$R/paper_2609_29395_amd/profile_summary.py copy`",
             "* `rocprofv3 --pmc WRITE_SIZE --output-format csv -d $O/cwrite -o run -- python "
             "$R/paper_2609_29395_amd/profile_summary.py copy`",
             f"* `python -m paper_2609_29395_amd.profile_summary traffic $O/pfetch $O/pwrite "
             f"$O/cfetch $O/cwrite {workload} {os.path.relpath(out_md, ROOT)}`", "",
             f"Calibration: a {COPY_MIB} MiB device copy reads FETCH_SIZE = {f_fac:.4f} x and WRITE_SIZE = "
             f"{w_fac:.4f} x its size; counters are divided by these factors.",
             "The figures also sit in `profile.json` with the hash of each kernel's source file when taken; "
             "bench.py reports traffic = null for a kernel whose source changed since.", "",
             "| kernel | launches | FETCH KiB/launch | WRITE KiB/launch | HBM MB/launch (calibrated) |",
             "|---|---|---|---|---|"]
    for k, v in sorted(out.items(), key=lambda kv: -kv[1]["bytes_per_launch"]):
        lines.append(f"| {k} | {v['launches']} | {v['fetch_kib']:.0f} | {v['write_kib']:.0f} | "
                     f"{v['bytes_per_launch'] / 1e6:.1f} |")
    lines.append("")
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))
    _update_profile(workload, "traffic", out)


def gemm_reference(out_md):
    """hipBLASLt (torch.matmul, bf16) on the plain GEMMs with the shapes of the
    16-cluster workload's convolutions, for comparison with the implicit-GEMM
    kernels: M = pixels of all replicas, N = output channels, K = 9 * input
    channels."""
    import torch
    shapes = [("256->256 conv as one GEMM", 524288, 256, 2304), ("64->256 conv", 524288, 256, 576),
              ("32->64 conv (32x32 images)", 2097152, 64, 288)]
    lines = ["# hipBLASLt reference on the convolution GEMM shapes", "",
             f"Command: `python -m paper_2609_29395_amd.profile_summary gemm-ref {out_md}`", "",
             "torch.matmul in bf16 (hipBLASLt), 10 timed calls after 3 warm-up calls, hipEvents.", "",
             "| shape | M | N | K | us | TFLOP/s |", "|---|---|---|---|---|---|"]
    for name, M, N, K in shapes:
        a = torch.randn(M, K, device="cuda", dtype=torch.bfloat16)
        b = torch.randn(K, N, device="cuda", dtype=torch.bfloat16)
        for _ in range(3):
            a @ b
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(10):
            a @ b
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / 10
        lines.append(f"| {name} | {M} | {N} | {K} | {ms * 1e3:.1f} | {2 * M * N * K / ms / 1e9:.1f} |")
        del a, b
    lines.append("")
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))


def layer_table(trace_dir, out_md, cmd):
    """Per-dispatch durations of one step (the third), in launch order."""
    rows = list(csv.DictReader(open(_one(os.path.join(trace_dir, "**", "*kernel_trace.csv")))))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    starts = [i for i, r in enumerate(rows) if "sample_kernel" in r["Kernel_Name"]]
    i0, i1 = starts[2], starts[3]
    lines = ["# One step, dispatch by dispatch", "", f"Command: `{' '.join(cmd)}`", "",
             "| # | kernel (label) | workgroups | us |", "|---|---|---|---|"]
    tot = 0.0
    for k, r in enumerate(rows[i0:i1]):
        d = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        tot += d
        wg = int(r["Grid_Size_X"]) // max(1, int(r["Workgroup_Size_X"]))
        lines.append(f"| {k} | {kernel_label(r['Kernel_Name'])} | {wg} | {d:.1f} |")
    lines += ["", f"Sum of kernel time in the step: {tot / 1e3:.3f} ms", ""]
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))


if __name__ == "__main__":
    what = sys.argv[1]
    if what == "copy":
        copy()
    elif what == "gemm-ref":
        gemm_reference(sys.argv[2])
    elif what == "layers":
        layer_table(sys.argv[2], sys.argv[3], sys.argv[4:])
    elif what == "stats":
        stats(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5:])
    elif what == "mfma":
        mfma(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5:])
    elif what == "traffic":
        traffic(*sys.argv[2:8])
    else:
        raise SystemExit(__doc__)
