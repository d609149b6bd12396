"""Summaries of rocprofv3 output for the kernels of this library.

  python -m paper_2609_29395_amd.profile_summary copy [--mib N] [--reps R]
      Run a plain device copy of a known size (the calibration kernel for the
      FETCH_SIZE / WRITE_SIZE counters).
  python -m paper_2609_29395_amd.profile_summary stats TRACE_DIR OUT.md CMD...
      Write a Markdown summary of `rocprofv3 --kernel-trace --stats` CSV output.
  python -m paper_2609_29395_amd.profile_summary traffic FETCH_DIR WRITE_DIR COPY_FETCH_DIR COPY_WRITE_DIR WORKLOAD OUT.json
  python -m paper_2609_29395_amd.profile_summary layers TRACE_DIR OUT.md CMD...
      Per-dispatch table of one step from `rocprofv3 --kernel-trace` CSV output.
  python -m paper_2609_29395_amd.profile_summary gemm-ref OUT.md
      hipBLASLt bf16 GEMMs of the convolution shapes, for comparison.
      Combine two counter runs of the workload (FETCH_SIZE, then WRITE_SIZE)
      into HBM bytes per launch for every kernel, each counter scaled by what
      it reads for the copy of known size (runs COPY_FETCH_DIR, COPY_WRITE_DIR).
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
                  r"(, (true|false))?>", name)
    if m:
        kind = "conv_fwd" if m.group(5) == "0" else "conv_dgrad"
        w = int(m.group(3)) * int(m.group(4))
        mode = "halo" if m.group(8) == "true" else "lds"
        kt = 192 if (mode == "halo" and m.group(2) == "64") else 64  # tap-row k tiles
        return f"{kind}<bf16,{m.group(1)}x{m.group(2)}x{kt},w{w},{mode}>"
    m = re.search(r"conv_img_kernel<(\d+), (\d+), (\d)>", name)
    if m:
        kind = "conv_fwd" if m.group(3) == "0" else "conv_dgrad"
        return f"{kind}<bf16,256x{m.group(2)}x{9 * int(m.group(1))},w8,img>"
    if re.search(r"wgrad_col_kernel", name):
        return "conv_wgrad<bf16,32x32,w4,col>"
    if re.search(r"conv_col_kernel", name):
        return "conv_fwd<bf16,256x32x32,w4,col>"
    if re.search(r"wgrad_img_kernel<", name):
        return "conv_wgrad<bf16,64x288,w8,img>"
    if re.search(r"wgrad_halo_kernel<", name):
        return "conv_wgrad<bf16,128x576,w8,halo>"
    m = re.search(r"wgrad_lds_kernel<(\d+), (\d+), (\d+), (\d+), (?:\d+, \d+, )?(true|false)>", name)
    if m:
        w = int(m.group(3)) * int(m.group(4))
        return f"conv_wgrad<bf16,{m.group(1)}x{m.group(2)},w{w},lds>"
    if re.search(r"wgrad_reduce2?_kernel", name):
        return "wgrad_reduce"  # the timing label of both widths
    m = re.search(r"::(\w+?)(_kernel)?[<(]", name)
    return m.group(1) if m else name


CSRC = os.path.join(ROOT, "paper_2609_29395_amd", "csrc")
SHARED_HEADERS = ("common.h",)  # device helpers every kernel source includes


def kernel_source(label: str) -> str:
    """The source file that holds the kernel a timing label names."""
    if label.startswith("conv_wgrad<") and label.endswith((",lds>", ",halo>", ",img>", ",col>")):
        return "k_wgrad_lds.hip"
    if label.startswith("conv_") and label.endswith((",lds>", ",halo>")):
        return "k_conv_lds.hip"
    if label.startswith("conv_") and label.endswith((",img>", ",col>")):
        return "k_conv_img.hip"
    if label.startswith("conv_"):
        return "k_conv.hip"
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


def stats(trace_dir, out_md, cmd):
    rows = list(csv.DictReader(open(_one(os.path.join(trace_dir, "**", "*kernel_stats.csv")))))
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    # instantiations that share a label (e.g. the head conv that also writes
    # the pooled features) are one row, as in the library's own timing
    by = collections.defaultdict(lambda: [0, 0.0])
    for r in rows:
        v = by[kernel_label(r["Name"])]
        v[0] += int(r["Calls"])
        v[1] += float(r["TotalDurationNs"])
    lines = [f"# Kernel time summary", "", f"Command: `{' '.join(cmd)}`", "",
             "| kernel (label) | calls | total ms | avg us | % |", "|---|---|---|---|---|"]
    for lab, (calls, tot) in sorted(by.items(), key=lambda kv: -kv[1][1]):
        lines.append(f"| {lab} | {calls} | {tot / 1e6:.3f} | {tot / calls / 1e3:.2f} | {100 * tot / total:.2f} |")
    lines += ["", f"Sum of kernel time: {total / 1e6:.3f} ms", ""]
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))


def _counter_per_dispatch(d, counter):
    rows = list(csv.DictReader(open(_one(os.path.join(d, "**", "*counter_collection.csv")))))
    per = collections.defaultdict(list)
    for r in rows:
        if r["Counter_Name"] == counter:
            per[r["Kernel_Name"]].append(float(r["Counter_Value"]))
    return per


def traffic(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, workload, out_json):
    fetch = _counter_per_dispatch(fetch_dir, "FETCH_SIZE")
    write = _counter_per_dispatch(write_dir, "WRITE_SIZE")
    expect_kib = COPY_MIB * 1024.0
    samples = lambda per: [v for vs in per.values() for v in vs if v > 0.25 * expect_kib]
    cf = samples(_counter_per_dispatch(copy_fetch_dir, "FETCH_SIZE"))
    cw = samples(_counter_per_dispatch(copy_write_dir, "WRITE_SIZE"))
    f_fac = (sum(cf) / len(cf)) / expect_kib if cf else 1.0
    w_fac = (sum(cw) / len(cw)) / expect_kib if cw else 1.0
    out = {"source_hashes": source_hashes(), "copy_mib": COPY_MIB, "fetch_factor": f_fac,
           "write_factor": w_fac, "kernels": {}}
    # per label: the launches of every instantiation with that label
    fl, wl = collections.defaultdict(list), collections.defaultdict(list)
    for k, v in fetch.items():
        fl[kernel_label(k)] += v
    for k, v in write.items():
        wl[kernel_label(k)] += v
    for k in set(fl) | set(wl):
        fv, wv = fl.get(k, []), wl.get(k, [])
        fk = sum(fv) / len(fv) if fv else 0.0
        wk = sum(wv) / len(wv) if wv else 0.0
        out["kernels"][f"{workload}:{k}"] = {
            "launches": max(len(fv), len(wv)), "fetch_kib": fk, "write_kib": wk,
            "bytes_per_launch": 1024.0 * (fk / f_fac + wk / w_fac)}
    with open(out_json, "w") as fh:
        json.dump(out, fh, indent=1, sort_keys=True)
    md = os.path.join(os.path.dirname(out_json), f"{workload}_traffic.md")
    lines = [f"# HBM traffic per launch, {workload}", "",
             "Commands (R = repository root; B = `python $R/bench.py --steps 5 --warmup 2 --timing-steps 2 "
             "--no-cpu-baseline --no-schedule-control --no-hbm-probes`):", "",
             "* `rocprofv3 --pmc FETCH_SIZE --output-format csv -d $R/gpurun_out/pfetch -o run -- $B`",
             "* `rocprofv3 --pmc WRITE_SIZE --output-format csv -d $R/gpurun_out/pwrite -o run -- $B`",
             "* `rocprofv3 --pmc FETCH_SIZE --output-format csv -d $R/gpurun_out/cfetch -o run -- python "
             "$R/paper_2609_29395_amd/profile_summary.py copy`",
             "* `rocprofv3 --pmc WRITE_SIZE --output-format csv -d $R/gpurun_out/cwrite -o run -- python "
             "$R/paper_2609_29395_amd/profile_summary.py copy`",
             f"* `python -m paper_2609_29395_amd.profile_summary traffic gpurun_out/pfetch gpurun_out/pwrite "
             f"gpurun_out/cfetch gpurun_out/cwrite {workload} {out_json}`", "",
             f"Calibration: a {COPY_MIB} MiB device copy reads FETCH_SIZE = {f_fac:.4f} x and WRITE_SIZE = "
             f"{w_fac:.4f} x its size; counters are divided by these factors.",
             "Kernel source hashes when taken: per kernel source file in `traffic.json` (`source_hashes`); "
             "bench.py reports traffic = null for a kernel whose source file changed since.", "",
             "| kernel | launches | FETCH KiB/launch | WRITE KiB/launch | HBM MB/launch (calibrated) |",
             "|---|---|---|---|---|"]
    for k, v in sorted(out["kernels"].items(), key=lambda kv: -kv[1]["bytes_per_launch"]):
        lines.append(f"| {k.split(':', 1)[1]} | {v['launches']} | {v['fetch_kib']:.0f} | {v['write_kib']:.0f} | "
                     f"{v['bytes_per_launch'] / 1e6:.1f} |")
    lines.append("")
    with open(md, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))


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
        stats(sys.argv[2], sys.argv[3], sys.argv[4:])
    elif what == "traffic":
        traffic(*sys.argv[2:8])
    else:
        raise SystemExit(__doc__)
