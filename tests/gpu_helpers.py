"""Shared plumbing of the GPU tests: seeded inputs, oracle expectations, device
upload and the calls through the C ABI binding."""
import os
import sys

import numpy as np

import oracle
from paper_2609_20186_amd import workloads as W

ORACLE_THREADS = max(1, min(16, os.cpu_count() or 1))
INT_KEYS = ("match_n", "match_end", "copy_len", "copy_tokens", "use_copy", "dtok", "dpar", "dn",
            "amax", "accept_len", "accept_node", "bonus", "out_tokens")
Z_TOL = 1e-3   # absolute tolerance on the probe logit


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def ocfg(lens, kappa, k, theta, n_cand=1):
    return oracle.make_cfg(lens, kappa, k, theta, n_cand)


def planted_workload(name, batch=None):
    """Inputs of a named workload with logits planted for the draft the oracle
    selects (steps 1-3), as the workload recipe prescribes."""
    wl = W.WORKLOADS[name]
    d = W.generate(wl, batch=batch)
    cfg = ocfg(wl.ngram_lens, wl.kappa, wl.k, wl.theta, wl.n_cand)
    sel = oracle.front(d["tokens"], d["lengths"], d["hidden"], d["w"], d["bias"], d["ntok"],
                       d["npar"], d["nn"], cfg)
    d["target"] = W.plant_batch(wl, d, sel)
    d["cfg"] = dict(lens=wl.ngram_lens, kappa=wl.kappa, k=wl.k, theta=wl.theta,
                    n_cand=wl.n_cand)
    return d


def oracle_step(d, rows=None):
    c = d["cfg"]
    cfg = ocfg(c["lens"], c["kappa"], c["k"], c["theta"], c.get("n_cand", 1))
    sl = slice(None) if rows is None else rows
    npar = None if d["npar"] is None else d["npar"][sl]
    T = d.get("T", 0.0)
    un = d["uniforms"][sl] if T > 0 else None
    ql = d.get("draft_logits")
    ua = d.get("accept_uniforms")
    return oracle.step(d["tokens"][sl], d["lengths"][sl], d["hidden"][sl], d["w"], d["bias"],
                       d["ntok"][sl], npar, d["nn"][sl], d["logits"][sl], cfg,
                       threads=ORACLE_THREADS, temperature=T, uniforms=un,
                       draft_logits=None if ql is None else ql[sl],
                       accept_uniforms=None if ua is None else ua[sl])


def to_device(d):
    import torch
    dev = {"tokens": torch.from_numpy(np.ascontiguousarray(d["tokens"])).cuda(),
           "lengths": torch.from_numpy(np.ascontiguousarray(d["lengths"])).cuda(),
           "hidden": torch.from_numpy(np.ascontiguousarray(d["hidden"]).view(np.int16)).cuda(),
           "w": torch.from_numpy(np.ascontiguousarray(d["w"])).cuda(),
           "ntok": torch.from_numpy(np.ascontiguousarray(d["ntok"])).cuda(),
           "npar": None if d["npar"] is None else
           torch.from_numpy(np.ascontiguousarray(d["npar"])).cuda(),
           "nn": torch.from_numpy(np.ascontiguousarray(d["nn"])).cuda(),
           "logits": torch.from_numpy(np.ascontiguousarray(d["logits"]).view(np.int16)).cuda(),
           "bias": float(d["bias"])}
    if d.get("T", 0.0) > 0:
        dev["uniforms"] = torch.from_numpy(
            np.ascontiguousarray(d["uniforms"], dtype=np.uint64).view(np.int64)).cuda()
    if d.get("draft_logits") is not None:
        dev["draft_logits"] = torch.from_numpy(
            np.ascontiguousarray(d["draft_logits"]).view(np.int16)).cuda()
        dev["accept_uniforms"] = torch.from_numpy(
            np.ascontiguousarray(d["accept_uniforms"], dtype=np.uint64).view(np.int64)).cuda()
    return dev


def with_temperature(d, T, seed):
    """The same inputs at sampling temperature T with seeded row uniforms."""
    d = dict(d)
    d["T"] = float(T)
    B, R = d["ntok"].shape
    d["uniforms"] = np.random.default_rng(seed).integers(0, 2 ** 64, (B, R), dtype=np.uint64)
    return d


def sd_cfg(d):
    from paper_2609_20186_amd import binding as sd
    c = d["cfg"]
    return sd.make_cfg(c["lens"], c["kappa"], c["k"], c["theta"], c.get("n_cand", 1))


def gpu_step(dev, d, mode=0, out=None, ws=None, sws=None):
    import torch
    from paper_2609_20186_amd import binding as sd
    B, R = dev["ntok"].shape
    k, W = d["cfg"]["k"], d["cfg"].get("n_cand", 1)
    out = out or sd.alloc_outputs(B, R, k, W)
    ws = ws if ws is not None else sd.alloc_workspace(B, R, dev["tokens"].shape[1], W)
    T = d.get("T", 0.0)
    if T > 0 and sws is None:
        sws = sd.alloc_sample_workspace(B, R, dev["logits"].shape[2])
    args = sd.build_step_args(dev, out, sd_cfg(d), mode, T, dev.get("uniforms"), sws,
                              draft_logits=dev.get("draft_logits"),
                              accept_uniforms=dev.get("accept_uniforms"))
    sd.switchsd_step(args, ws)
    torch.cuda.synchronize()
    res = {k2: v.cpu().numpy() for k2, v in out.items()}
    return res, ws


def gpu_stages(dev, d):
    """The four stage entry points in order."""
    import torch
    from paper_2609_20186_amd import binding as sd
    B, R = dev["ntok"].shape
    k, W = d["cfg"]["k"], d["cfg"].get("n_cand", 1)
    cfg = sd_cfg(d)
    o = sd.alloc_outputs(B, R, k, W)
    ws = sd.alloc_workspace(B, R, dev["tokens"].shape[1], W)
    sd.switchsd_ngram_match(dev["tokens"], dev["lengths"], cfg, o["match_n"], o["match_end"],
                            o["copy_len"], o["copy_tokens"], ws)
    sd.switchsd_probe_score(dev["hidden"], dev["w"], dev["bias"], o["z"])
    sd.switchsd_select_draft(o["match_n"], o["copy_len"], o["copy_tokens"], o["z"], dev["ntok"],
                             dev["npar"], dev["nn"], cfg, o["use_copy"], o["dtok"], o["dpar"],
                             o["dn"])
    T = d.get("T", 0.0)
    if T > 0:
        # the stage entry point verifies every sequence with q when given (the
        # step keeps copy drafts one-hot); with q the drafts are chains and
        # dpar is not passed
        q = dev.get("draft_logits")
        sd.switchsd_verify_sample(dev["logits"], T, dev["uniforms"], o["dtok"],
                                  None if q is not None else o["dpar"],
                                  o["dn"], o["accept_len"], o["accept_node"], o["bonus"],
                                  o["out_tokens"], o["amax"], ws,
                                  sd.alloc_sample_workspace(B, R, dev["logits"].shape[2]),
                                  draft_logits=dev.get("draft_logits"),
                                  accept_uniforms=dev.get("accept_uniforms"))
    else:
        sd.switchsd_verify_accept(dev["logits"], o["dtok"], o["dpar"], o["dn"],
                                  o["accept_len"], o["accept_node"], o["bonus"],
                                  o["out_tokens"], o["amax"], ws)
    torch.cuda.synchronize()
    return {k2: v.cpu().numpy() for k2, v in o.items()}, ws


def assert_match(got, exp, rows=None, what=""):
    sl = slice(None) if rows is None else rows
    for key in INT_KEYS:
        g = got[key][sl]
        e = exp[key]
        if key == "copy_tokens":
            g = g.reshape(e.shape)
        if not np.array_equal(g, e):
            bad = np.argwhere(g != e)[:5]
            raise AssertionError(f"{what}: {key} differs at {bad.tolist()}: "
                                 f"gpu {g[tuple(bad[0])]} oracle {e[tuple(bad[0])]}")
    dz = np.abs(got["z"][sl].astype(np.float64) - exp["z"].astype(np.float64))
    assert dz.max(initial=0.0) <= Z_TOL, f"{what}: |dz| = {dz.max()}"
