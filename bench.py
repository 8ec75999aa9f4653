#!/usr/bin/env python3
"""Benchmark of SwitchSD's speculation-control step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload C2]

One step = one call of ``switchsd_step`` over the whole batch: suffix n-gram
match, probe, copy/neural switch, verify-argmax and accept for all B
sequences, inputs resident in HBM.  The default workload is the Llama-3-8B
shaped copy-heavy batch (B=32, L=4096, V=128256, d=4096, k=7).  Input sets
are rotated so that more than 512 MB is touched between two uses of one set:
the 256 MB Infinity Cache cannot serve a step from the previous one.

Prints ONE JSON line (steps/s, ms/step, the dominant kernel against the HBM
roofline, the verify-argmax rate, and the CPU oracle timed on a bounded sample
of the same workload on this host).  ``--workload C2W10`` measures the paper's
multi-candidate copy setting (W = 10 candidates of D = 20 tokens, R = 201).
"""
import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2609_20186_amd import workloads as W  # noqa: E402

HBM_PEAK_GBPS = 8000.0
# VALU issue rate: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz (a wave64 op takes 4
# cycles on one SIMD) = 39.3 T lane-ops/s; one FMA is one op here
VALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12
# VALU ops per logit of the draw at T > 0: about 1.5 in the row-maximum pass
# and 19.3 in the sum pass (the compiled chunk loop of k_sample_sums issues 617
# VALU instructions per 32 logits of a lane: unpack, subtract, scale, clamp,
# rint, reduce, 6 fused multiply-adds, convert, ldexp, floor, widen to
# binary64, accumulate, and the wave sums)
SAMPLE_OPS_PER_LOGIT = 20.8
METRIC = "speculation-control steps/s + verify-argmax HBM GB/s (% peak), B=32 V=128256"
PROFILES = os.path.join(ROOT, "profiles")
ROTATE_BYTES = 512 << 20


def kernel_sha():
    from paper_2609_20186_amd.profile_summary import kernel_sha as sha
    return sha()


def algorithmic_bytes(wl, rows_read, d_sel=None):
    """Bytes one step must move at least: each context token once, the hidden
    states and probe weight, every logits row it reads, the neural draft and
    the outputs."""
    B, R, k, Wc = wl.B, wl.R, wl.k, max(1, wl.n_cand)
    ins = B * wl.L * 4 + B * 4 + B * wl.d * 2 + wl.d * 4 + B * R * 4 + B * 4
    if not wl.chain:
        ins += B * R * 4
    logits = int(np.sum(rows_read)) * wl.V * 2
    # match_n, match_end [W], copy_len [W], copy_tokens [W, k], z, use_copy, dtok,
    # dpar, dn, amax, accept_len, accept_node, bonus, out_tokens
    outs = B * 4 + 2 * B * Wc * 4 + B * Wc * k * 4 + B * 4 * 2 + B * R * 4 * 2 + B * 4 + \
        B * R * 4 + B * 4 * 3 + B * R * 4
    return ins + logits + outs, logits


def resolve_mode(wl, mode):
    """The launch the library's AUTO mode picks (switchsd_step)."""
    if mode:
        return mode
    cn = 1 + max(1, wl.n_cand) * wl.k
    return 1 if cn >= wl.R and wl.R <= 64 else 2


def upload(d):
    import torch
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    return {"tokens": t(d["tokens"]), "lengths": t(d["lengths"]),
            "hidden": t(d["hidden"].view(np.int16)), "w": t(d["w"]), "ntok": t(d["ntok"]),
            "npar": None if d["npar"] is None else t(d["npar"]), "nn": t(d["nn"]),
            "logits": t(d["logits"].view(np.int16)), "bias": float(d["bias"])}


def plant_with_library(wl, d, sd):
    """Plant the logits for the drafts the library itself selects (its split
    step's front half writes the draft before any row is read)."""
    import torch
    dev = upload(d)
    out = sd.alloc_outputs(wl.B, wl.R, wl.k, wl.n_cand)
    ws = sd.alloc_workspace(wl.B, wl.R, wl.L, wl.n_cand)
    cfg = sd.make_cfg(wl.ngram_lens, wl.kappa, wl.k, wl.theta, wl.n_cand)
    sd.switchsd_step(sd.build_step_args(dev, out, cfg, sd.MODE_SPLIT), ws)
    torch.cuda.synchronize()
    sel = {k: out[k].cpu().numpy() for k in ("dtok", "dpar", "dn", "use_copy")}
    W.plant_batch(wl, d, sel)
    return sel


def host_cores():
    """Cores this process may run on (its affinity mask), and what the host
    reports in all."""
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count() or 1
    return max(1, usable), os.cpu_count() or usable


def cpu_baseline(wl_name, budget_s):
    """The oracle as it stands, on this host, over whole steps of the same
    workload (inputs generated and planted on the CPU): once with one thread
    per usable core and once with one thread, each repeated for about half of
    `budget_s` seconds."""
    import oracle
    wl = W.WORKLOADS[wl_name]
    d = W.generate(wl)
    cfg = oracle.make_cfg(wl.ngram_lens, wl.kappa, wl.k, wl.theta, wl.n_cand)
    sel = oracle.front(d["tokens"], d["lengths"], d["hidden"], d["w"], d["bias"], d["ntok"],
                       d["npar"], d["nn"], cfg)
    W.plant_batch(wl, d, sel)
    args = (d["tokens"], d["lengths"], d["hidden"], d["w"], d["bias"], d["ntok"], d["npar"],
            d["nn"], d["logits"], cfg)
    usable, reported = host_cores()

    def timed(threads, seconds):
        n = 0
        t0 = time.perf_counter()
        while True:
            oracle.step(*args, threads=threads)
            n += 1
            el = time.perf_counter() - t0
            if el >= seconds or n >= 100000:
                return n, el

    n, el = timed(usable, budget_s / 2)
    n1, el1 = timed(1, budget_s / 2)
    return {"value": n / el, "unit": "steps/s", "cores": usable, "kind": "oracle",
            "sample": f"{n} whole {wl_name} steps (B={wl.B}, all sequences) in {el:.1f} s on "
                      f"{usable} threads (the cores of this process's affinity mask; the host "
                      f"reports {reported})",
            "single_thread": {"value": n1 / el1, "unit": "steps/s", "cores": 1,
                              "sample": f"{n1} whole {wl_name} steps in {el1:.1f} s"},
            "host_cpu_count": reported}


def draft_distribution(wl, d, sets, T, torch):
    """Draft logits for --draft-q (the target's plus N(0, 0.5) noise, one
    device copy per rotation set) with the neural drafts' tokens drawn from
    softmax(q / T) row by row (written into every set), and the accept
    uniforms."""
    rng = np.random.default_rng(20187)
    lf = (d["logits"].astype(np.uint32) << 16).view(np.float32)
    q = W.f32_to_bf16_bits((lf + rng.normal(0, 0.5, lf.shape)).astype(np.float32))
    qf = (q.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    ntok = d["ntok"].copy()
    for b in range(wl.B):
        for r in range(wl.R - 1):
            z = (qf[b, r] - qf[b, r].max()) / T
            pr = np.exp(z)
            ntok[b, r + 1] = int(rng.choice(wl.V, p=pr / pr.sum()))
    nt = torch.from_numpy(ntok).cuda()
    for st in sets:
        st["ntok"].copy_(nt)
    qd = torch.from_numpy(q.view(np.int16)).cuda()
    qdev = [qd] + [qd.clone() for _ in range(len(sets) - 1)]
    uacc = torch.from_numpy(rng.integers(0, 2 ** 64, (wl.B, wl.R), dtype=np.uint64)
                            .view(np.int64)).cuda()
    return qdev, uacc


_CALIB = None


def calibrate_lib():
    """The measurement library (streaming-read calibration, delay kernel)."""
    global _CALIB
    if _CALIB is None:
        import ctypes
        from paper_2609_20186_amd import build as hb
        _CALIB = ctypes.CDLL(hb.CALIBRATE_LIB)
        _CALIB.switchsd_calibrate_delay.argtypes = [ctypes.c_double, ctypes.c_void_p]
        _CALIB.switchsd_calibrate_read.argtypes = [ctypes.c_void_p, ctypes.c_int64,
                                                   ctypes.c_int32, ctypes.c_int32,
                                                   ctypes.c_void_p, ctypes.c_void_p]
        _CALIB.switchsd_calibrate_read_dyn.argtypes = [ctypes.c_void_p, ctypes.c_int64,
                                                       ctypes.c_int32, ctypes.c_int32,
                                                       ctypes.c_void_p, ctypes.c_void_p,
                                                       ctypes.c_void_p]
    return _CALIB


def event_timings(torch, stream, fn, n, reps):
    """`reps` runs of fn over n calls, back to back on `stream` between two
    HIP events each: ms per call of every run.  Before each run a delay
    kernel holds the stream (25 us per call, at least 0.5 ms) while the n
    calls are queued from the host, so that they run back to back: the timed
    region holds exactly the n calls and the GPU gaps between them, not the
    host's launch rate."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    lib = calibrate_lib()
    per = []
    host = []
    for _ in range(reps):
        torch.cuda.synchronize()
        if lib.switchsd_calibrate_delay(min(500.0 + 25.0 * n, 2e5), stream.cuda_stream):
            raise RuntimeError("switchsd_calibrate_delay failed")
        e0.record(stream)
        t0 = time.perf_counter()
        fn(0, n)
        host.append((time.perf_counter() - t0) / n * 1e6)
        e1.record(stream)
        torch.cuda.synchronize()
        per.append(e0.elapsed_time(e1) / n)
    event_timings.host_us = float(np.median(host))
    return per


def read_calibration(torch, stream, sets, nbytes, cus):
    """The streaming-read calibration kernel over the same rotated logits
    (each launch reads `nbytes` of the next copy), back to back: a sweep of
    work-groups per CU and chunks in flight, its best point, and the same
    read without rotation (one copy, which the 256 MB Infinity Cache can
    hold between launches)."""
    lib = calibrate_lib()
    out = torch.empty(16 * cus, dtype=torch.int32, device="cuda")
    sp = stream.cuda_stream
    ptrs = [st["logits"].data_ptr() for st in sets]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(wg, depth, rotate, n=300, src=None, nb=None):
        srcs = [src] if src is not None else (ptrs if rotate else ptrs[:1])
        nb = nbytes if nb is None else nb

        def fn(n_):
            for i in range(n_):
                rc = lib.switchsd_calibrate_read(srcs[i % len(srcs)], nb, wg, depth,
                                                 out.data_ptr(), sp)
                if rc:
                    raise RuntimeError(f"switchsd_calibrate_read returned {rc}")
        fn(20)
        torch.cuda.synchronize()
        lib.switchsd_calibrate_delay(min(500.0 + 25.0 * n, 2e5), sp)
        e0.record(stream)
        fn(n)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n * 1e3

    def timed_dyn(wg, static_pct, n=300):
        ctr = torch.zeros((n + 20) * 128, dtype=torch.int32, device="cuda")

        def fn(i0, n_):
            for i in range(i0, i0 + n_):
                rc = lib.switchsd_calibrate_read_dyn(ptrs[i % len(ptrs)], nbytes, wg, static_pct,
                                                     ctr.data_ptr() + 512 * i, out.data_ptr(),
                                                     sp)
                if rc:
                    raise RuntimeError(f"switchsd_calibrate_read_dyn returned {rc}")
        fn(0, 20)
        torch.cuda.synchronize()
        lib.switchsd_calibrate_delay(min(500.0 + 25.0 * n, 2e5), sp)
        e0.record(stream)
        fn(20, n)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n * 1e3

    dyn = []
    for per_cu in (2, 4):
        for pct in (0, 50, 75, 90):
            dyn.append({"workgroups": per_cu * cus, "static_percent": pct,
                        "us": round(timed_dyn(per_cu * cus, pct), 2)})

    sweep = []
    for per_cu in (1, 2, 4, 8):
        for depth in (2, 3, 4):
            us = timed(per_cu * cus, depth, True)
            sweep.append({"workgroups": per_cu * cus, "depth": depth, "us": round(us, 2)})
    best = min(sweep, key=lambda r: r["us"])
    us2 = next(r["us"] for r in sweep if r["workgroups"] == 2 * cus and r["depth"] == 2)
    cached = timed(2 * cus, 2, False)
    # the asymptotic rate: one 1 GiB read per launch (no cache can hold it)
    big = torch.empty(1 << 30, dtype=torch.uint8, device="cuda").fill_(1)
    big_us = min(timed(w, dp, False, 20, big.data_ptr(), 1 << 30)
                 for w in (4 * cus, 8 * cus) for dp in (2, 3))
    del big
    gb = lambda us: round(nbytes / (us * 1e-6) / 1e9, 1)  # noqa: E731
    return {"bytes": nbytes, "kernel": "read_calibration.hip: 16-byte nontemporal loads, 16 KB "
                                       "chunks per 256-lane work-group, back to back over the "
                                       "rotated copies",
            "best": {**best, "GBps": gb(best["us"]),
                     "frac": round(gb(best["us"]) / HBM_PEAK_GBPS, 4)},
            "step_kernel_shape": {"workgroups": 2 * cus, "depth": 2, "us": us2, "GBps": gb(us2)},
            "one_GiB_read": {"us": round(big_us, 1),
                             "GBps": round((1 << 30) / (big_us * 1e-6) / 1e9, 1),
                             "frac": round((1 << 30) / (big_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)},
            "unrotated_same_shape": {"us": round(cached, 2), "GBps": gb(cached),
                                     "note": "one copy re-read each launch: the Infinity Cache "
                                             "serves part of it"},
            "sweep": sweep,
            "claims_sweep": dyn}


def decode_loop(args, wl, d, sets, cfg, sd, torch, T, uni, sws):
    """K steps with commit captured in one HIP graph, cycling over the input
    copies (the contexts, lengths and draft-model positions are shared and
    grow); each replay starts from the initial contexts (restored outside the
    timed region)."""
    K = args.loop
    B, R = wl.B, wl.R
    Lmax = wl.L + K * R
    tokens = torch.zeros((B, Lmax), dtype=torch.int32, device="cuda")
    tokens[:, :wl.L] = sets[0]["tokens"]
    lengths0 = sets[0]["lengths"].clone()
    lengths = lengths0.clone()
    draft_pos = lengths0.clone()
    lag = torch.zeros(B, dtype=torch.int32, device="cuda")
    tokens0 = tokens.clone()
    nset = len(sets)
    outs = [sd.alloc_outputs(B, R, wl.k, wl.n_cand) for _ in range(nset)]
    ws = sd.alloc_workspace(B, R, Lmax, wl.n_cand)
    args_l = []
    for st, o in zip(sets, outs):
        inp = dict(st)
        inp["tokens"], inp["lengths"] = tokens, lengths
        args_l.append(sd.build_step_args(inp, o, cfg, args.mode, T, uni, sws, draft_pos, lag))

    def run_steps():
        for i in range(K):
            sd.switchsd_step(args_l[i % nset], ws)

    def reset():
        tokens.copy_(tokens0)
        lengths.copy_(lengths0)
        draft_pos.copy_(lengths0)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run_steps()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    eager_len = lengths.clone()
    reset()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run_steps()
    reps = max(3, args.steps // K)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    total = 0.0
    for rep in range(reps + 1):
        reset()
        torch.cuda.synchronize()
        e0.record()
        graph.replay()
        e1.record()
        torch.cuda.synchronize()
        if rep > 0:                      # the first replay is a warm-up
            total += e0.elapsed_time(e1)
        assert torch.equal(lengths, eager_len), "graph replay disagrees with the eager loop"
    us = total / reps / K * 1e3
    grown = (eager_len - lengths0).float().mean().item()
    return {"steps_per_graph": K, "replays": reps, "us_per_step": round(us, 2),
            "steps_per_s": round(1e6 / us, 1),
            "tokens_appended_per_sequence_per_step": round(grown / K, 3),
            "note": "contexts grow in place; inputs cycle over the rotation copies"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", default="C2", choices=sorted(W.WORKLOADS))
    ap.add_argument("--mode", type=int, default=0, help="0 auto, 1 fused, 2 split")
    ap.add_argument("--temperature", type=float, default=0.0,
                    help="> 0: verification draws the rows' tokens at this sampling "
                         "temperature (App. A) with seeded uniforms")
    ap.add_argument("--loop", type=int, default=0,
                    help="also time the decode loop: this many steps with commit (append "
                         "the accepted tokens, draft-model lag) captured in one HIP graph")
    ap.add_argument("--labels", type=int, default=0,
                    help="also time the copy-mode labels (Sec. 3.2) of the workload's "
                         "contexts with this window length n (the paper's is 5)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--repeats", type=int, default=5,
                    help="timed runs of --steps steps each; the line reports their median")
    ap.add_argument("--draft-q", action="store_true",
                    help="at T > 0, verify the neural drafts by speculative sampling with a "
                         "draft distribution q (draft logits = the target's plus N(0, 0.5) "
                         "noise, drafted tokens drawn from q)")
    ap.add_argument("--no-calibration", action="store_true",
                    help="skip the streaming-read calibration of the logits' size")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="after timing, run a plain device copy of this many MB five times "
                         "(the reference kernel for scaling HBM counters)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the speculation-control step shards by sequence with "
              "no exchange between GPUs, so one GPU's throughput is the measure. Use --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_20186_amd import binding as sd

    wl = W.WORKLOADS[args.workload]
    print(f"[bench] generating {wl.name} inputs", file=sys.stderr, flush=True)
    d = W.generate(wl)
    sel = plant_with_library(wl, d, sd)

    base = upload(d)
    # bytes one step reads (the drafted rows for a split step, every row the
    # fused launch reads otherwise): enough copies that > 512 MB lie between
    # two uses of one copy
    cn = 1 + max(1, wl.n_cand) * wl.k
    if resolve_mode(wl, args.mode) == sd.MODE_FUSED:
        rows0 = np.maximum(np.clip(d["nn"], 1, wl.R), cn) if cn < wl.R else np.full(wl.B, wl.R)
    else:
        rows0 = sel["dn"]
    step_bytes = int(np.sum(rows0)) * wl.V * 2 + d["tokens"].nbytes + d["hidden"].nbytes
    nrot = max(1, math.ceil(ROTATE_BYTES / step_bytes))
    sets = [base] + [{k: (v.clone() if hasattr(v, "clone") else v) for k, v in base.items()}
                     for _ in range(nrot - 1)]
    cfg = sd.make_cfg(wl.ngram_lens, wl.kappa, wl.k, wl.theta, wl.n_cand)
    outs = [sd.alloc_outputs(wl.B, wl.R, wl.k, wl.n_cand) for _ in range(nrot)]
    ws = sd.alloc_workspace(wl.B, wl.R, wl.L, wl.n_cand)
    T = args.temperature
    qdev = uacc = None
    if T > 0:
        uni = torch.from_numpy(np.random.default_rng(20186).integers(
            0, 2 ** 64, (wl.B, wl.R), dtype=np.uint64).view(np.int64)).cuda()
        sws = sd.alloc_sample_workspace(wl.B, wl.R, wl.V)
        if args.draft_q:
            qdev, uacc = draft_distribution(wl, d, sets, T, torch)
        step_args = [sd.build_step_args(s, o, cfg, args.mode, T, uni, sws,
                                        draft_logits=None if qdev is None else qdev[i],
                                        accept_uniforms=uacc)
                     for i, (s, o) in enumerate(zip(sets, outs))]
    else:
        step_args = [sd.build_step_args(s, o, cfg, args.mode) for s, o in zip(sets, outs)]
    import ctypes
    lib = sd.lib
    stream = torch.cuda.current_stream()
    sptr = stream.cuda_stream
    wsp, wsn = ws.data_ptr(), ws.numel()
    refs = [ctypes.byref(a) for a in step_args]

    def run(i0, n):
        for i in range(i0, i0 + n):
            rc = lib.switchsd_step(refs[i % nrot], wsp, wsn, sptr)
            if rc:
                raise sd.SwitchsdError("switchsd_step", rc)

    run(0, args.warmup)
    # exactly --steps steps per timed run, --repeats runs; the reported figure
    # is their median; then each step bracketed by its own events
    per_step = event_timings(torch, stream, run, args.steps, max(1, args.repeats))
    host_us = event_timings.host_us
    ms = float(np.median(per_step))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    # every rotation set that ran must agree with the first (same inputs, same
    # outputs); small workloads have more sets than steps
    o0 = {k: v.cpu() for k, v in outs[0].items()}
    for o in outs[1:min(nrot, max(args.warmup, args.steps))]:
        for k, v in o.items():
            assert torch.equal(v.cpu(), o0[k]), f"rotation set disagrees on {k}"

    mode = resolve_mode(wl, args.mode)
    cn = 1 + max(1, wl.n_cand) * wl.k
    if mode == sd.MODE_FUSED:
        rows_read = np.maximum(np.clip(d["nn"], 1, wl.R), cn) if cn < wl.R \
            else np.full(wl.B, wl.R)
    else:
        rows_read = sel["dn"]
    alg, alg_logits = algorithmic_bytes(wl, rows_read)
    step_gbps = alg / (ms * 1e-3) / 1e9

    # verification alone (stage entry point), rows of the chosen draft
    if T > 0:
        vargs = [(st["logits"].data_ptr(), wl.B, wl.R, wl.V, T, uni.data_ptr(),
                  None if qdev is None else qdev[i].data_ptr(),
                  None if uacc is None else uacc.data_ptr(),
                  o["dtok"].data_ptr(), None if qdev is not None else o["dpar"].data_ptr(),
                  o["dn"].data_ptr(),
                  o["accept_len"].data_ptr(), o["accept_node"].data_ptr(), o["bonus"].data_ptr(),
                  o["out_tokens"].data_ptr(), o["amax"].data_ptr(), wsp, wsn, sws.data_ptr(),
                  sws.numel(), sptr) for i, (st, o) in enumerate(zip(sets, outs))]
        vfn, vname = lib.switchsd_verify_sample, "switchsd_verify_sample"
    else:
        vargs = [(st["logits"].data_ptr(), wl.B, wl.R, wl.V, o["dtok"].data_ptr(),
                  o["dpar"].data_ptr(), o["dn"].data_ptr(), o["accept_len"].data_ptr(),
                  o["accept_node"].data_ptr(), o["bonus"].data_ptr(),
                  o["out_tokens"].data_ptr(), o["amax"].data_ptr(), wsp, wsn, sptr)
                 for st, o in zip(sets, outs)]
        vfn, vname = lib.switchsd_verify_accept, "switchsd_verify_accept"

    def run_verify(i0, n):
        for i in range(i0, i0 + n):
            rc = vfn(*vargs[i % nrot])
            if rc:
                raise sd.SwitchsdError(vname, rc)

    nv = max(200, args.steps // 4)
    run_verify(0, 20)
    v_per = event_timings(torch, stream, run_verify, nv, max(1, args.repeats))
    vms = float(np.median(v_per))
    vbytes = int(np.sum(sel["dn"])) * wl.V * 2
    v_gbps = vbytes / (vms * 1e-3) / 1e9

    loop_res = None
    if args.loop > 0:
        loop_res = decode_loop(args, wl, d, sets, cfg, sd, torch, T,
                               uni if T > 0 else None, sws if T > 0 else None)

    label_res = None
    if args.labels > 0:
        lab = torch.empty(base["tokens"].shape, dtype=torch.uint8, device="cuda")
        lws = torch.zeros(max(sd.label_workspace_bytes(wl.B, wl.L), 256), dtype=torch.uint8,
                          device="cuda")
        for _ in range(3):
            sd.switchsd_copy_labels(base["tokens"], base["lengths"], args.labels, lab, lws)
        torch.cuda.synchronize()
        nl = 20
        e0.record(stream)
        for _ in range(nl):
            sd.switchsd_copy_labels(base["tokens"], base["lengths"], args.labels, lab, lws)
        e1.record(stream)
        torch.cuda.synchronize()
        lus = e0.elapsed_time(e1) / nl * 1e3
        label_res = {"n": args.labels, "us_per_call": round(lus, 1),
                     "positions_per_s": round(wl.B * wl.L / (lus * 1e-6), 1),
                     "copy_mode_share": round(float(lab.float().mean().item()), 4)}

    if args.copy_calibration_mb > 0:
        n = args.copy_calibration_mb << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # the dominant kernel: the fused launch, or the verify launch of a split
    # step; at T > 0 the verification's launches together.  `achieved` divides
    # the algorithmic bytes (ops) of one launch (call) by its own duration,
    # each launch bracketed by its own HIP events on the launch stream
    launch_ms = ms
    # the row maxima launch also takes the q rows unless it streams long
    # drafts (and, in the step, unless there are several copy candidates)
    listed = wl.R > 64 and wl.B <= 256 and wl.V % 8 == 0
    q_merged_verify = qdev is not None and not listed
    q_merged = (qdev is not None and max(1, wl.n_cand) == 1 and
                not (mode == sd.MODE_SPLIT and listed))
    if T > 0:
        qrows = 0 if qdev is None else int(np.sum(np.clip(sel["dn"] - 1, 0, None) *
                                                  (sel["use_copy"] == 0)))
        ops = (vbytes / 2 + qrows * wl.V) * SAMPLE_OPS_PER_LOGIT
        dom = {"kernel": ("sampled verification (row maxima of p and q, then weight sums with "
                          "the accept tests, then the residual draw: 3 launches)"
                          if q_merged_verify else
                          "sampled verification (row maxima, q row maxima, weight sums with the "
                          "accept tests, residual draw: 4 launches)"
                          if qdev is not None else
                          "sampled verification (row maxima, then weight sums with the draw: "
                          "2 launches)"),
               "bound": "alu", "unit": "TOP/s (VALU lane-ops)", "peak": round(VALU_PEAK_TOPS, 1),
               "gbps": ops / (vms * 1e-3) / 1e12, "bytes": int(ops), "ms": vms,
               "traffic_file": f"traffic_sampled_verify_{wl.name}.json"}
    elif mode == sd.MODE_FUSED:
        dom = {"kernel": "k_switchsd (fused step)", "gbps": alg / (launch_ms * 1e-3) / 1e9,
               "bytes": alg, "ms": launch_ms,
               "traffic_file": f"traffic_fused_step_{wl.name}.json"}
    else:
        # long drafts of up to 256 sequences with 16-byte aligned rows: the
        # streamed verify kernel; short drafts of at most one sequence per CU:
        # the polling verify kernel; otherwise the step kernel's argmax role
        streamed = wl.R > 64 and wl.B <= 256 and wl.V % 8 == 0
        cus = torch.cuda.get_device_properties(0).multi_processor_count
        kname = ("k_verify_stream" if streamed else
                 "k_verify_poll" if wl.R <= 64 and wl.B <= cus else "k_switchsd")
        dom = {"kernel": f"{kname} (verify launch of the split step)",
               "gbps": vbytes / (vms * 1e-3) / 1e9, "bytes": vbytes, "ms": vms,
               "traffic_file": f"traffic_verify_{wl.name}.json"}
    calib = None
    if not args.no_calibration and T == 0:
        cus = torch.cuda.get_device_properties(0).multi_processor_count
        nb = int(np.sum(rows_read if mode == sd.MODE_FUSED else sel["dn"])) * wl.V * 2 // 16 * 16
        calib = read_calibration(torch, stream, sets, nb, cus)
    traffic = None
    tf = os.path.join(PROFILES, dom["traffic_file"])
    if os.path.exists(tf):
        with open(tf) as f:
            tr = json.load(f)
        if tr.get("kernel_sha") == kernel_sha() and tr.get("workload") == wl.name:
            traffic = tr.get("hbm_bytes_per_launch")

    res = {
        "metric": METRIC, "value": round(1e3 / ms, 1), "unit": "steps/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: B={wl.B} L={wl.L} V={wl.V} d={wl.d} k={wl.k} R={wl.R}"
                               f" W={max(1, wl.n_cand)} ngram={list(wl.ngram_lens)}"
                               f" kappa={wl.kappa}" + (f" T={T}" if T > 0 else ""),
                   "global_batch": wl.B, "seq_len": wl.L, "parallelism": "none (1 GPU)",
                   "launch": {1: "fused, 1 kernel", 2: "split, 2 kernels"}[mode] +
                             ("" if T <= 0 else
                              " + 1 kernel for the weight sums and the draw at T > 0"
                              if qdev is None else
                              (" (with the q row maxima)" if q_merged else
                               " + 1 kernel for the q row maxima") +
                              " + 2 kernels for the weight sums with the accept tests and the"
                              " residual draw"),
                   "rotation_sets": nrot},
        "roofline": {"bound": dom.get("bound", "hbm"), "achieved": round(dom["gbps"], 1),
                     "peak": dom.get("peak", HBM_PEAK_GBPS), "unit": dom.get("unit", "GB/s"),
                     "frac": round(dom["gbps"] / dom.get("peak", HBM_PEAK_GBPS), 4),
                     "traffic": traffic, "kernel": dom["kernel"],
                     ("algorithmic_ops_per_call" if T > 0 else "algorithmic_bytes_per_launch"):
                         dom["bytes"]},
        "timing": {"repeats": len(per_step), "steps_per_repeat": args.steps,
                   "ms_per_step_median": round(ms, 5),
                   "ms_per_step_min": round(float(np.min(per_step)), 5),
                   "ms_per_step_max": round(float(np.max(per_step)), 5),
                   "host_us_per_launch": round(host_us, 2),
                   "note": "value, ms_per_step and roofline.achieved: the median of the "
                           "repeats, each --steps launches between two HIP events on the "
                           "launch stream, queued behind a delay kernel so that they run "
                           "back to back (GPU launch gaps included, host launch rate not)"},
        "step_GBps": round(step_gbps, 1),
        ("verify_sampled" if T > 0 else "verify_argmax"):
            {"GBps": round(v_gbps, 1), "frac": round(v_gbps / HBM_PEAK_GBPS, 4),
             "us_per_call": round(vms * 1e3, 2),
             "us_per_call_min": round(float(np.min(v_per)) * 1e3, 2),
             "us_per_call_max": round(float(np.max(v_per)) * 1e3, 2), "bytes_per_call": vbytes,
             # the whole [B, R, V] tensor over the same time: what the call costs
             # per byte a caller hands over (rows past a draft are never read)
             "tensor_bytes": wl.B * wl.R * wl.V * 2,
             "tensor_GBps_effective": round(wl.B * wl.R * wl.V * 2 / (vms * 1e-3) / 1e9, 1)},
        "copy_fraction": round(float(np.mean(sel["use_copy"])), 3),
        "mean_accept_len": round(float(o0["accept_len"].float().mean()), 3),
        "kernel_sha": kernel_sha(),
    }
    if calib:
        res["read_calibration"] = calib
    if qdev is not None:
        res["config"]["draft_distribution"] = ("q: the target's logits plus N(0, 0.5), drafted "
                                               "tokens drawn from q (speculative sampling)")
    if loop_res:
        res["decode_loop"] = loop_res
    if label_res:
        res["copy_labels"] = label_res
    if not args.no_cpu:
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(wl.name, args.cpu_seconds)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
