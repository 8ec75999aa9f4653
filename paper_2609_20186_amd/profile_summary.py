"""Summarize rocprofv3 CSV output of ``bench.py`` into ``profiles/``.

    python -m paper_2609_20186_amd.profile_summary trace  <dir> <out.md> "<command>"
    python -m paper_2609_20186_amd.profile_summary traffic <fetch_dir> <write_dir> <copy_mb> \\
        <out.md> <out.json> "<fetch command>" "<write command>" [<workload> <kernel> <label>]

``trace`` reads a ``--kernel-trace --stats`` run and lists per-kernel
dispatch counts and durations.  ``traffic`` reads two ``--pmc`` runs
(FETCH_SIZE, then WRITE_SIZE, KiB per dispatch), scales both by what the same
counters read for the plain device copy of ``copy_mb`` MB that
``bench.py --copy-calibration-mb`` runs, and writes the HBM bytes per launch
of the named kernel (default: the fused step kernel ``k_switchsd`` of C2; the
largest grid of that kernel dispatched at least 10 times), with the hash of the kernel
source the counters were taken on, so that ``bench.py`` drops the figure once
the kernel changes.
"""
import csv
import glob
import hashlib
import json
import os
import re
import statistics
import sys

COPY = "copyBuffer"


def _rows(d, pattern):
    files = glob.glob(os.path.join(d, "**", pattern), recursive=True)
    if not files:
        raise SystemExit(f"no {pattern} under {d}")
    out = []
    for f in files:
        with open(f, newline="") as fh:
            out.extend(csv.DictReader(fh))
    return out


def kernel_sha():
    """Hash of the code (comments and blank space dropped) of the kernels, their
    launch configuration and the constants they share: a counter reading stays
    valid while none of these changes."""
    h = hashlib.sha256()
    csrc = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc")
    for name in ("switchsd_kernels.hip", "switchsd_api.cpp", "switchsd_internal.h"):
        with open(os.path.join(csrc, name)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def trace(d, out, cmd):
    rows = _rows(d, "*kernel_trace.csv")
    by = {}
    for r in rows:
        name = r["Kernel_Name"]
        grid = int(r.get("Grid_Size", r.get("Grid_Size_X", 0)) or 0)
        wg = int(r.get("Workgroup_Size", r.get("Workgroup_Size_X", 1)) or 1)
        dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        by.setdefault((name, grid // max(wg, 1)), []).append(dur)
    lines = [f"# Kernel trace: {os.path.basename(out)[:-3]}", "", f"Command: `{cmd}`", "",
             "| kernel | work-groups | dispatches | median us | mean us | min us | max us |",
             "|---|---|---|---|---|---|---|"]
    for (name, wgs), ds in sorted(by.items(), key=lambda kv: -sum(kv[1])):
        short = name.replace("(anonymous namespace)::", "").split("(")[0][-60:]
        lines.append(f"| `{short}` | {wgs} | {len(ds)} | {statistics.median(ds):.2f} | "
                     f"{statistics.mean(ds):.2f} | {min(ds):.2f} | {max(ds):.2f} |")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _counter(d, counter, kernel):
    rows = _rows(d, "*counter_collection.csv")
    k, c = [], []
    for r in rows:
        if r.get("Counter_Name") != counter:
            continue
        v = float(r["Counter_Value"])
        name = r["Kernel_Name"]
        # plain or templated (k_switchsd<false, false>) instantiations
        if kernel + "(" in name or kernel + "<" in name or name.endswith(kernel):
            grid = int(r.get("Grid_Size", 0) or 0)
            k.append((grid, v))
        elif COPY in r["Kernel_Name"]:
            c.append(v)
    return k, c


def traffic(fdir, wdir, copy_mb, out_md, out_json, fcmd, wcmd, workload="C2",
            kernel="k_switchsd", label="fused step kernel"):
    copy_bytes = copy_mb << 20
    kf, cf = _counter(fdir, "FETCH_SIZE", kernel)
    kw, cw = _counter(wdir, "WRITE_SIZE", kernel)
    # the kernel's largest grid dispatched at least 10 times: the timed launch
    # (the fused step is larger than the benchmark's verify-only launches)
    grids = {}
    for g, _ in kf:
        grids[g] = grids.get(g, 0) + 1
    g = max(gg for gg, n in grids.items() if n >= 10)
    fetch_kib = statistics.median([v for gg, v in kf if gg == g])
    write_kib = statistics.median([v for gg, v in kw if gg == g])
    copy_fetch = statistics.median(sorted(cf)[-5:])   # the large calibration copies
    copy_write = statistics.median(sorted(cw)[-5:])
    sf = copy_fetch * 1024 / copy_bytes
    sw = copy_write * 1024 / copy_bytes
    fetch_b = fetch_kib * 1024 / sf
    write_b = write_kib * 1024 / sw
    res = {"workload": workload, "kernel": kernel, "kernel_sha": kernel_sha(), "grid_threads": g,
           "fetch_kib_per_launch": fetch_kib, "write_kib_per_launch": write_kib,
           "copy_mb": copy_mb, "copy_fetch_kib": copy_fetch, "copy_write_kib": copy_write,
           "fetch_scale": sf, "write_scale": sw,
           "hbm_bytes_per_launch": int(round(fetch_b + write_b))}
    with open(out_json, "w") as f:
        json.dump(res, f, indent=1)
    lines = [f"# HBM traffic: {label} (`{kernel}`), {workload}", "",
             f"FETCH_SIZE command: `{fcmd}`", "", f"WRITE_SIZE command: `{wcmd}`", "",
             "| quantity | value |", "|---|---|",
             f"| {label} FETCH_SIZE per dispatch | {fetch_kib:.0f} KiB |",
             f"| {label} WRITE_SIZE per dispatch | {write_kib:.1f} KiB |",
             f"| plain copy of {copy_mb} MB: FETCH_SIZE | {copy_fetch:.0f} KiB (scale {sf:.4f}) |",
             f"| plain copy of {copy_mb} MB: WRITE_SIZE | {copy_write:.0f} KiB (scale {sw:.4f}) |",
             f"| scaled HBM bytes per launch (read + write) | {fetch_b + write_b:,.0f} B |",
             f"| kernel code sha256[:16] (comments dropped) | {res['kernel_sha']} |"]
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


if __name__ == "__main__":
    if sys.argv[1] == "trace":
        trace(sys.argv[2], sys.argv[3], sys.argv[4])
    else:
        traffic(sys.argv[2], sys.argv[3], int(sys.argv[4]), sys.argv[5], sys.argv[6],
                sys.argv[7], sys.argv[8], *sys.argv[9:12])
