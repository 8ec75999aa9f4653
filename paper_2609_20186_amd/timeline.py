"""Per-phase timeline of the fused step (measurement support).

    python -m paper_2609_20186_amd.timeline --workload C2 [--launches 30] [--out file.md]

Runs the step through ``libswitchsd_timeline.so`` -- the same sources as the
library, compiled with per-work-group stamps of the GPU's 100 MHz real-time
clock at the end of each phase -- over rotated copies of the workload's inputs
(more than 512 MB between two uses of one copy), and prints, as the median
over the launches, when each phase ends relative to the first work-group's
start: the scan tiles, the front (match, probe, switch, draft), the argmax
row segments, the sequences' last arrivals (or, where the epilogue polls the
segment results, when it has seen all of them, and how many poll rounds that
took) and the accept epilogues.  The
stamps cost a few stores per work-group.
"""
import argparse
import ctypes
import math
import os
import sys

import numpy as np

from . import binding as sd
from . import build as B
from . import workloads as W

ROLE = {0: "scan", 1: "probe", 2: "argmax"}
TICKS_PER_US = 100.0        # s_memrealtime runs at 100 MHz


def _upload(d, torch):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    return {"tokens": t(d["tokens"]), "lengths": t(d["lengths"]),
            "hidden": t(d["hidden"].view(np.int16)), "w": t(d["w"]), "ntok": t(d["ntok"]),
            "npar": None if d["npar"] is None else t(d["npar"]), "nn": t(d["nn"]),
            "logits": t(d["logits"].view(np.int16)), "bias": float(d["bias"])}


def _q(a, f):
    return float(np.quantile(a, f)) if len(a) else float("nan")


def analyse(st, B_):
    """Phase statistics (us after the earliest start) of one launch; st is the
    [grid, 8] array of stamps."""
    start = st[:, 0].astype(np.int64)
    t0 = start.min()
    us = lambda v: (v.astype(np.int64) - t0) / TICKS_PER_US  # noqa: E731
    role = (st[:, 7] >> 32).astype(np.int64)
    seq = (st[:, 7] & 0xFFFFFFFF).astype(np.int64)
    out = {"last work-group start": us(start).max()}
    for r, name in ROLE.items():
        m = role == r
        if m.any():
            v = us(st[m, 1])
            out[f"{name} work-groups done (median)"] = _q(v, 0.5)
            out[f"{name} work-groups done (p90)"] = _q(v, 0.9)
            out[f"{name} work-groups done (last)"] = v.max()
    fr = st[:, 2] != 0
    if fr.any():
        v = us(st[fr, 2])
        out["front done (median)"] = _q(v, 0.5)
        out["front done (last)"] = v.max()
    ar = st[:, 3] != 0
    if ar.any():
        last_arr = np.array([us(st[ar & (seq == b), 3]).max() for b in range(B_)
                             if (ar & (seq == b)).any()])
        out["sequence's last arrival (median)"] = _q(last_arr, 0.5)
        out["sequence's last arrival (last)"] = last_arr.max()
    polled = (st[:, 6] >> 32) != 0     # the accept epilogue polled the segment results
    el = (st[:, 5] != 0) & ~polled
    if el.any():
        v = us(st[el, 5])
        out["accept epilogue's loads returned (median)"] = _q(v, 0.5)
        out["accept epilogue's loads returned (last)"] = v.max()
    if polled.any():
        v = us(st[polled, 5])
        out["accept poll started (median)"] = _q(v, 0.5)
        out["accept poll started (last)"] = v.max()
        rounds = (st[polled, 6] >> 32).astype(np.int64) - 1
        out["accept poll rounds (median)"] = _q(rounds, 0.5)
        out["accept poll rounds (max)"] = rounds.max()
    tiles = (st[:, 6] & 0xFFFFFFFF) != 0
    if tiles.any():
        rounds = (st[tiles, 6] & 0xFFFFFFFF).astype(np.int64) - 1
        out["tile poll rounds (median)"] = _q(rounds, 0.5)
        out["tile poll rounds (max)"] = rounds.max()
    am = role == 2
    if am.any():
        # work-groups are dispatched to the 8 XCDs in turn (block index mod 8)
        blk = np.nonzero(am)[0]
        done = us(st[am, 1])
        per = [np.median(done[blk % 8 == x]) for x in range(8) if (blk % 8 == x).any()]
        out["argmax done, median per XCD (fastest)"] = min(per)
        out["argmax done, median per XCD (slowest)"] = max(per)
        half = len(blk) // 2
        out["argmax done, first half of the dispatch (median)"] = _q(done[:half], 0.5)
        out["argmax done, second half of the dispatch (median)"] = _q(done[half:], 0.5)
    ep = st[:, 4] != 0
    if ep.any():
        v = us(st[ep, 4])
        out["accept epilogue done (median)"] = _q(v, 0.5)
        out["accept epilogue done (last)"] = v.max()
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="C2", choices=sorted(W.WORKLOADS))
    ap.add_argument("--launches", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--out", default="")
    args = ap.parse_args()
    import torch
    lib = ctypes.CDLL(B.TIMELINE_LIB)
    lib.switchsd_step.argtypes = [ctypes.POINTER(sd.StepArgs), ctypes.c_void_p, ctypes.c_size_t,
                                  ctypes.c_void_p]
    lib.switchsd_timeline_buffer.argtypes = [ctypes.c_void_p]
    lib.switchsd_timeline_buffer.restype = None
    wl = W.WORKLOADS[args.workload]
    print(f"[timeline] generating {wl.name} inputs", file=sys.stderr, flush=True)
    d = W.generate(wl)
    cfg = sd.make_cfg(wl.ngram_lens, wl.kappa, wl.k, wl.theta, wl.n_cand)
    # plant the logits for the drafts the library selects (its split step's front)
    base = _upload(d, torch)
    out = sd.alloc_outputs(wl.B, wl.R, wl.k, wl.n_cand)
    ws = sd.alloc_workspace(wl.B, wl.R, wl.L, wl.n_cand)
    sd.switchsd_step(sd.build_step_args(base, out, cfg, sd.MODE_SPLIT), ws)
    torch.cuda.synchronize()
    W.plant_batch(wl, d, {k: out[k].cpu().numpy() for k in ("dtok", "dpar", "dn", "use_copy")})
    base = _upload(d, torch)
    nrot = max(1, math.ceil((512 << 20) / d["logits"].nbytes))
    sets = [base] + [{k: (v.clone() if hasattr(v, "clone") else v) for k, v in base.items()}
                     for _ in range(nrot - 1)]
    outs = [sd.alloc_outputs(wl.B, wl.R, wl.k, wl.n_cand) for _ in range(nrot)]
    argl = [sd.build_step_args(s, o, cfg, sd.MODE_FUSED) for s, o in zip(sets, outs)]
    stream = torch.cuda.current_stream().cuda_stream
    wsp, wsn = ws.data_ptr(), ws.numel()

    def step(i):
        rc = lib.switchsd_step(ctypes.byref(argl[i % nrot]), wsp, wsn, stream)
        if rc:
            raise sd.SwitchsdError("switchsd_step", rc)

    for i in range(args.warmup):
        step(i)
    # the fused grid: probe and scan work-groups, then B * R rows of
    # ceil(2 * CUs / (B * R)) segments at most
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    rows_ = wl.B * wl.R
    grid = wl.B * (math.ceil(wl.L / 1024) + 1) + rows_ + 2 * cus + 64
    bufs = torch.zeros((args.launches, grid, 8), dtype=torch.int64, device="cuda")
    torch.cuda.synchronize()
    for i in range(args.launches):
        lib.switchsd_timeline_buffer(bufs[i].data_ptr())
        step(args.warmup + i)
    lib.switchsd_timeline_buffer(None)
    torch.cuda.synchronize()
    stamps = bufs.cpu().numpy().view(np.uint64)
    rows = []
    for i in range(args.launches):
        st = stamps[i]
        st = st[st[:, 0] != 0]
        rows.append(analyse(st, wl.B))
    keys = list(rows[0].keys())
    lines = [f"# Timeline of the fused step, {wl.name}", "",
             f"Command: `python -m paper_2609_20186_amd.timeline --workload {wl.name} "
             f"--launches {args.launches}`", "",
             f"Launch grid: {int((stamps[0][:, 0] != 0).sum())} work-groups; "
             f"{args.launches} launches over {nrot} rotated input copies; times in us after "
             f"the first work-group's start (100 MHz clock, 0.01 us resolution), median over "
             f"the launches (min - max in brackets).", "",
             "| phase | us |", "|---|---|"]
    for k in keys:
        v = np.array([r[k] for r in rows if k in r])
        lines.append(f"| {k} | {np.median(v):.2f} ({v.min():.2f} - {v.max():.2f}) |")
    text = "\n".join(lines) + "\n"
    print(text)
    if args.out:
        with open(args.out, "w") as f:
            f.write(text)


if __name__ == "__main__":
    main()
