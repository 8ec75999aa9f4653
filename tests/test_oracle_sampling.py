"""Pins of the oracle's draw at sampling temperature T > 0 (App. A).

The draws are pinned to mathematics computed here independently of the
oracle's arithmetic: exact softmax probabilities (numpy exp in float64), the
T -> 0 limit (the greedy argmax, itself pinned elsewhere), the T -> infinity
limit (uniform), hand-derived fixture cases, and the speculative-sampling
property for a one-hot draft (accept with probability p(x), else the emitted
token follows the residual p without x).
"""
import json
import os

import numpy as np
import pytest

import brute
import oracle
from paper_2609_20186_amd.workloads import f32_to_bf16_bits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _cases():
    with open(os.path.join(GOLDEN, "sample_cases.jsonl")) as f:
        return [json.loads(s) for s in f if s.strip()]


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c["why"][:40])
def test_golden_sample(case):
    row = np.array([int(h, 16) for h in case["row"]], np.uint16)
    assert oracle.sample_row(row, case["T"], case["u"]) == case["expect"]


def test_weight_is_two_to_the_t():
    """w = trunc(2^20 * 2^t) up to the polynomial's relative error, with t the
    float32 value (l - m) * c; t < -24 gives 0."""
    rng = np.random.default_rng(31)
    for T in (0.05, 0.3, 1.0, 2.5, 40.0):
        c = oracle.sample_scale(T)
        assert c == np.float32(np.log2(np.e) / T)
        m = np.float32(rng.normal(3, 2))
        for l in np.float32(m - rng.exponential(3.0, 400)):
            t = (np.float32(l) - m) * np.float32(c)         # float32 arithmetic
            w = oracle.sample_weight(l, m, c)
            if t < -24:
                assert w == 0
                continue
            exact = 2.0 ** (20 + float(t))
            assert exact * (1 - 3e-7) - 1 <= w <= exact * (1 + 3e-7), (T, l, m, w, exact)


def _boundaries(row, T):
    """u32 boundaries U_j where the draw changes from j-1 to j (bisection)."""
    V = row.size
    out = [0]
    for j in range(1, V):
        lo, hi = 0, 2 ** 32 - 1
        if oracle.sample_row(row, T, hi) < j:
            out.append(2 ** 32)
            continue
        while lo < hi:
            mid = (lo + hi) // 2
            if oracle.sample_row(row, T, mid) >= j:
                hi = mid
            else:
                lo = mid + 1
        out.append(lo)
    out.append(2 ** 32)
    return np.array(out, np.float64)


@pytest.mark.parametrize("T", [0.3, 1.0, 3.0])
def test_draw_is_inverse_cdf_of_softmax(T):
    """The draw is monotone in u and the share of u values giving index j is
    softmax(l / T)_j, computed here in float64, within the fixed-point error."""
    rng = np.random.default_rng(32)
    for _ in range(6):
        V = int(rng.integers(2, 12))
        row = f32_to_bf16_bits(rng.normal(0, 1.5, V).astype(np.float32))
        lf = brute.bf16_to_f32(row).astype(np.float64)
        p = np.exp((lf - lf.max()) / T)
        p /= p.sum()
        U = _boundaries(row, T)
        share = np.diff(U) / 2.0 ** 32
        assert np.all(np.diff(U) >= 0)
        np.testing.assert_allclose(share, p, atol=2e-6 * V + 1e-6, rtol=2e-6)


def test_cold_limit_is_greedy():
    """T = 1e-4 with every other logit >= 0.01 below a unique maximum: every
    draw is the greedy argmax."""
    rng = np.random.default_rng(33)
    for _ in range(50):
        V = int(rng.integers(2, 300))
        f = rng.normal(0, 1, V).astype(np.float32)
        row = f32_to_bf16_bits(f)
        lf = brute.bf16_to_f32(row)
        top = int(np.argmax(lf))
        if np.sort(lf)[-2] > lf[top] - 0.01:
            continue
        for u in rng.integers(0, 2 ** 32, 20, dtype=np.uint64):
            assert oracle.sample_row(row, 1e-4, int(u)) == top == brute.argmax_row(row)


def test_hot_limit_is_uniform():
    """T = 1e6: every weight is 2^20, so index j takes u in [j 2^32 / V, (j+1) 2^32 / V)."""
    rng = np.random.default_rng(34)
    for V in (3, 7, 100):
        row = f32_to_bf16_bits(rng.normal(0, 1, V).astype(np.float32))
        for u in rng.integers(0, 2 ** 32, 200, dtype=np.uint64):
            assert oracle.sample_row(row, 1e6, int(u)) == int(u) * V // 2 ** 32


def test_nan_never_drawn_and_degenerate_rows_greedy():
    rng = np.random.default_rng(35)
    row = f32_to_bf16_bits(rng.normal(0, 1, 50).astype(np.float32))
    row[::3] = 0x7FC0
    for u in rng.integers(0, 2 ** 32, 500, dtype=np.uint64):
        assert row[oracle.sample_row(row, 1.0, int(u))] != 0x7FC0
    allnan = np.full(9, 0x7FC0, np.uint16)
    neginf = np.array([0x7FC0, 0xFF80, 0xFF80], np.uint16)
    posinf = np.array([0x3F80, 0x7F80, 0x7F80], np.uint16)
    for r in (allnan, neginf, posinf):
        for u in (0, 2 ** 31, 2 ** 32 - 1):
            assert oracle.sample_row(r, 0.7, u) == brute.argmax_row(r)


def test_one_hot_speculative_sampling_property():
    """A single drafted token x after the anchor: over many uniforms the draft
    is accepted with probability p(x), and after a rejection the emitted token
    follows p restricted to tokens other than x (the residual of speculative
    sampling with a one-hot draft)."""
    rng = np.random.default_rng(36)
    V, T = 6, 0.8
    row = f32_to_bf16_bits(rng.normal(0, 1, V).astype(np.float32))
    lf = brute.bf16_to_f32(row).astype(np.float64)
    p = np.exp((lf - lf.max()) / T)
    p /= p.sum()
    x = int(np.argsort(p)[-2])
    n = 40000
    logits = np.zeros((n, 2, V), np.uint16)
    logits[:, 0] = row
    tokens = np.zeros((n, 4), np.int32)
    lengths = np.full(n, 1, np.int32)                      # no match: the neural draft is used
    ntok = np.full((n, 2), x, np.int32)
    cfg = oracle.make_cfg((1,), 1, 1, np.inf)
    res = oracle.step(tokens, lengths, np.zeros((n, 0), np.uint16), np.zeros(0, np.float32), 0.0,
                      ntok, None, np.full(n, 2, np.int32), logits, cfg, threads=8,
                      temperature=T, uniforms=rng.integers(0, 2 ** 32, (n, 2), dtype=np.uint32))
    acc = res["accept_len"] == 1
    assert abs(acc.mean() - p[x]) < 4 * np.sqrt(p[x] * (1 - p[x]) / n)
    rej = res["bonus"][~acc]
    q = p.copy()
    q[x] = 0
    q /= q.sum()
    freq = np.bincount(rej, minlength=V) / rej.size
    assert freq[x] == 0
    np.testing.assert_allclose(freq, q, atol=4 * np.sqrt(q.max() / rej.size) + 1e-3)


def test_step_at_temperature_uses_the_draws():
    """oracle.step at T > 0: each row's token is the per-row draw, and the
    accept result is the (pinned) accept walk over those tokens."""
    rng = np.random.default_rng(37)
    for _ in range(100):
        B, R, V = 3, int(rng.integers(2, 7)), int(rng.integers(2, 9))
        k = R - 1
        tokens = rng.integers(0, 3, (B, 30)).astype(np.int32)
        lengths = rng.integers(1, 31, B).astype(np.int32)
        logits = f32_to_bf16_bits(rng.normal(0, 1, (B, R, V)).astype(np.float32))
        un = rng.integers(0, 2 ** 32, (B, R), dtype=np.uint32)
        ntok = rng.integers(0, V, (B, R)).astype(np.int32)
        nn = rng.integers(1, R + 1, B).astype(np.int32)
        T = float(rng.choice([0.1, 0.7, 1.5]))
        cfg = oracle.make_cfg((2, 1), 1, k, 0.0)
        hid = np.zeros((B, 4), np.uint16)
        res = oracle.step(tokens, lengths, hid, np.zeros(4, np.float32), 0.0, ntok, None, nn,
                          logits, cfg, temperature=T, uniforms=un)
        for b in range(B):
            am = [oracle.sample_row(logits[b, r], T, un[b, r]) if r < res["dn"][b] else -1
                  for r in range(R)]
            assert res["amax"][b].tolist() == am
            exp = brute.accept(res["dtok"][b], res["dpar"][b], res["dn"][b], am, R)
            assert (res["accept_len"][b], res["accept_node"][b], res["bonus"][b]) == exp[:3]
            assert res["out_tokens"][b].tolist() == exp[3]
