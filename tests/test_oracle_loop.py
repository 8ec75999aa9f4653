"""Pins of the decode-loop bookkeeping (Sec. 3.3, KV Cache Synchronization):
hand-derived commits, invariants over random loops, and a loop whose final
context is rebuilt independently from the per-step outputs."""
import json
import os

import numpy as np
import pytest

import oracle
from paper_2609_20186_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _cases():
    with open(os.path.join(GOLDEN, "commit_cases.jsonl")) as f:
        return [json.loads(s) for s in f if s.strip()]


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c["why"][:40])
def test_golden_commit(case):
    x = np.array([case["x"]], np.int32)
    L = np.array([case["L"]], np.int32)
    dp = np.array([case["draft_pos"]], np.int32)
    R = len(case["out"])
    res = {"out_tokens": np.array([case["out"]], np.int32),
           "accept_len": np.array([case["accept_len"]], np.int32),
           "use_copy": np.array([case["use_copy"]], np.int32)}
    lag = oracle.commit(x, L, dp, res)
    assert x[0].tolist() == case["x_after"] and int(L[0]) == case["L_after"]
    assert int(dp[0]) == case["draft_pos_after"] and int(lag[0]) == case["lag"]
    assert R >= 1


def loop(wl_name, steps, extra, seed=0):
    """The oracle's decode loop: step, then commit, repeated; returns the
    initial and final state and the per-step outputs."""
    wl = W.WORKLOADS[wl_name]
    d = W.generate(wl)
    B = wl.B
    Lmax = wl.L + extra
    tokens = np.zeros((B, Lmax), np.int32)
    tokens[:, :wl.L] = d["tokens"]
    lengths = d["lengths"].copy()
    draft_pos = lengths.copy()
    cfg = oracle.make_cfg(wl.ngram_lens, wl.kappa, wl.k, wl.theta, wl.n_cand)
    init = (tokens.copy(), lengths.copy())
    hist = []
    for s in range(steps):
        res = oracle.step(tokens, lengths, d["hidden"], d["w"], d["bias"], d["ntok"], d["npar"],
                          d["nn"], d["logits"], cfg, threads=8)
        before = (lengths.copy(), draft_pos.copy())
        lag = oracle.commit(tokens, lengths, draft_pos, res)
        hist.append((res, before, lag))
    return init, (tokens, lengths, draft_pos), hist


def test_loop_invariants_and_rebuild():
    (t0, l0), (t1, l1, dp1), hist = loop("C1", 40, extra=100)
    Lmax = t0.shape[1]
    # the context is the initial prefix followed by each step's accepted
    # tokens and bonus, in order, cut at the capacity
    for b in range(t0.shape[0]):
        seq = list(t0[b, :l0[b]])
        for res, (lb, dpb), lag in hist:
            a = int(res["accept_len"][b])
            seq += [int(v) for v in res["out_tokens"][b, :a + 1]]
        seq = seq[:Lmax]
        assert int(l1[b]) == len(seq)
        assert t1[b, :l1[b]].tolist() == seq
    # draft position: unchanged by copy steps, L + accept after neural ones
    for res, (lb, dpb), lag in hist:
        for b in range(t0.shape[0]):
            a, uc = int(res["accept_len"][b]), int(res["use_copy"][b])
            Lnew = min(int(lb[b]) + a + 1, Lmax)
            exp_dp = int(dpb[b]) if uc else min(int(lb[b]) + a, Lnew)
            assert lag[b] == Lnew - exp_dp and 0 <= exp_dp <= Lnew
            if not uc and Lnew == int(lb[b]) + a + 1:
                assert lag[b] == 1                 # only the bonus is new to the drafter


def test_loop_lag_accumulates_over_copy_steps():
    rng = np.random.default_rng(40)
    for _ in range(200):
        Lmax = int(rng.integers(5, 60))
        x = np.zeros((1, Lmax), np.int32)
        L = np.array([int(rng.integers(1, Lmax))], np.int32)
        dp = np.array([int(rng.integers(0, L[0] + 1))], np.int32)
        lag_prev = int(L[0] - dp[0])
        for _ in range(6):
            a = int(rng.integers(0, 4))
            uc = int(rng.integers(0, 2))
            res = {"out_tokens": rng.integers(0, 9, (1, a + 1)).astype(np.int32),
                   "accept_len": np.array([a], np.int32), "use_copy": np.array([uc], np.int32)}
            L0 = int(L[0])
            lag = int(oracle.commit(x, L, dp, res)[0])
            grown = int(L[0]) - L0
            assert grown == min(a + 1, Lmax - L0)
            if uc:
                assert lag == lag_prev + grown
            lag_prev = lag
