"""Pins of the oracle's verification at sampling temperature T > 0 (App. A).

The draws are pinned to mathematics computed here independently of the
oracle's arithmetic: float64 softmax(l / T) at full vocabulary (total
variation), exact big-integer boundaries of the inverse CDF, the T -> 0 limit
(the greedy argmax, itself pinned elsewhere), the T -> infinity limit
(uniform), hand-derived fixture cases, the speculative-sampling property for a
one-hot draft, and, for drafts that carry their distribution q, the exact law
of the emitted token (computed with fractions from the oracle's own accept and
residual boundaries) against p.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import brute
import oracle
from paper_2609_20186_amd.workloads import f32_to_bf16_bits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TWO64 = 2 ** 64
# total variation between the normalized integer weights and float64 softmax
TV_BOUND = 1e-6


def _jsonl(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [json.loads(s) for s in f if s.strip()]


def _bits(h):
    return np.array([int(x, 16) for x in h], np.uint16)


def _softmax64(row, T):
    lf = brute.bf16_to_f32(row).astype(np.float64)
    p = np.exp((lf - lf.max()) / T)
    return p / p.sum()


def _u64(rng, shape):
    return rng.integers(0, 2 ** 64, shape, dtype=np.uint64)


@pytest.mark.parametrize("case", _jsonl("sample_cases.jsonl"), ids=lambda c: c["why"][:40])
def test_golden_sample(case):
    assert oracle.sample_row(_bits(case["row"]), case["T"], case["u"]) == case["expect"]


@pytest.mark.parametrize("case", _jsonl("spec_cases.jsonl"), ids=lambda c: c["why"][:40])
def test_golden_spec(case):
    p, q = _bits(case["p"]), _bits(case["q"])
    if "accept" in case:
        assert oracle.spec_accept(p, q, case["T"], case["x"], case["u"]) == case["accept"]
    else:
        assert oracle.residual_row(p, q, case["T"], case["u"]) == case["residual"]


def test_weight_is_two_to_the_forty_plus_t():
    """w = floor(2^40 * 2^t) up to the polynomial's relative error, with t the
    float32 value (l - m) * c; t < -41 gives 0."""
    rng = np.random.default_rng(31)
    for T in (0.05, 0.3, 1.0, 2.5, 40.0):
        c = oracle.sample_scale(T)
        assert c == np.float32(np.log2(np.e) / T)
        m = np.float32(rng.normal(3, 2))
        for l in np.float32(m - rng.exponential(6.0, 400)):
            t = (np.float32(l) - m) * np.float32(c)         # float32 arithmetic
            w = oracle.sample_weight(l, m, c)
            if t < -41:
                assert w == 0
                continue
            exact = 2.0 ** (40 + float(t))
            assert exact * (1 - 3e-7) - 1 <= w <= exact * (1 + 3e-7), (T, l, m, w, exact)


@pytest.mark.parametrize("V", [128256, 151936])
@pytest.mark.parametrize("planted", [False, True])
def test_weights_match_softmax_at_full_vocabulary(V, planted):
    """At the workloads' vocabularies, for N(0,1) rows (clamped to +-7.5 as the
    workloads draw them) with and without a planted +8 logit, the normalized
    integer weights are within total variation 1e-6 of float64 softmax(l / T)
    at T = 0.2, 0.7, 1.0 and 1.5."""
    rng = np.random.default_rng([V, planted])
    f = np.clip(rng.normal(0, 1, V), -7.5, 7.5).astype(np.float32)
    if planted:
        f[rng.integers(V)] = 8.0
    row = f32_to_bf16_bits(f)
    for T in (0.2, 0.7, 1.0, 1.5):
        w, Z = oracle.row_weights(row, T)
        assert Z == int(w.astype(object).sum())
        tv = 0.5 * np.abs(_softmax64(row, T) - w.astype(np.float64) / Z).sum()
        assert tv <= TV_BOUND, (V, planted, T, tv)


def _boundaries(fn, V):
    """Lowest 64-bit u at which fn(u) >= j, for j = 1..V-1 (bisection), with
    0 first and 2^64 last."""
    out = [0]
    for j in range(1, V):
        if fn(TWO64 - 1) < j:
            out.append(TWO64)
            continue
        lo, hi = 0, TWO64 - 1
        while lo < hi:
            mid = (lo + hi) // 2
            if fn(mid) >= j:
                hi = mid
            else:
                lo = mid + 1
        out.append(lo)
    out.append(TWO64)
    return out


def _ceil_div(a, b):
    return -(-a // b)


@pytest.mark.parametrize("T", [0.3, 1.0, 3.0])
def test_draw_is_exact_inverse_cdf(T):
    """The draw changes from j - 1 to j exactly at u = ceil(S_{j-1} 2^64 / Z)
    (S the prefix sums of the weights, in big integers here), so the share of
    u giving j is w_j / Z to within 2^-64; and it is softmax(l / T) within the
    weights' error."""
    rng = np.random.default_rng(32)
    for _ in range(6):
        V = int(rng.integers(2, 12))
        row = f32_to_bf16_bits(rng.normal(0, 1.5, V).astype(np.float32))
        w, Z = oracle.row_weights(row, T)
        S = np.cumsum([int(x) for x in w]).tolist()
        U = _boundaries(lambda u: oracle.sample_row(row, T, u), V)
        assert U == [0] + [_ceil_div(S[j - 1] * TWO64, Z) for j in range(1, V)] + [TWO64]
        share = np.diff(np.array(U, dtype=object)).astype(np.float64) / 2.0 ** 64
        np.testing.assert_allclose(share, _softmax64(row, T), atol=1e-6)


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
        for u in _u64(rng, 20):
            assert oracle.sample_row(row, 1e-4, int(u)) == top == brute.argmax_row(row)


def test_hot_limit_is_uniform():
    """T = 1e30: every t rounds P(t) to 1, every weight is 2^40, so index j
    takes u in [j 2^64 / V, (j+1) 2^64 / V)."""
    rng = np.random.default_rng(34)
    for V in (3, 7, 100):
        row = f32_to_bf16_bits(rng.normal(0, 1, V).astype(np.float32))
        w, Z = oracle.row_weights(row, 1e30)
        assert np.all(w == 2 ** 40) and Z == V * 2 ** 40
        for u in _u64(rng, 200):
            assert oracle.sample_row(row, 1e30, int(u)) == int(u) * V // TWO64


def test_nan_never_drawn_and_degenerate_rows_greedy():
    rng = np.random.default_rng(35)
    row = f32_to_bf16_bits(rng.normal(0, 1, 50).astype(np.float32))
    row[::3] = 0x7FC0
    for u in _u64(rng, 500):
        assert row[oracle.sample_row(row, 1.0, int(u))] != 0x7FC0
    allnan = np.full(9, 0x7FC0, np.uint16)
    neginf = np.array([0x7FC0, 0xFF80, 0xFF80], np.uint16)
    posinf = np.array([0x3F80, 0x7F80, 0x7F80], np.uint16)
    for r in (allnan, neginf, posinf):
        w, Z = oracle.row_weights(r, 0.7)
        g = brute.argmax_row(r)
        assert Z == 2 ** 40 and w[g] == 2 ** 40
        for u in (0, 2 ** 63, TWO64 - 1):
            assert oracle.sample_row(r, 0.7, u) == g


def test_one_hot_speculative_sampling_property():
    """A single drafted token x after the anchor: over many uniforms the draft
    is accepted with probability p(x), and after a rejection the emitted token
    follows p restricted to tokens other than x (the residual of speculative
    sampling with a one-hot draft)."""
    rng = np.random.default_rng(36)
    V, T = 6, 0.8
    row = f32_to_bf16_bits(rng.normal(0, 1, V).astype(np.float32))
    p = _softmax64(row, T)
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
                      temperature=T, uniforms=_u64(rng, (n, 2)))
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
        un = _u64(rng, (B, R))
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


# ---- drafts with their own distribution q (speculative sampling proper)

def _accept_threshold(prow, qrow, T, x):
    """The lowest u that rejects x (2^64: none), found by bisection; the test
    must be monotone in u."""
    thr = _boundaries(lambda u: 0 if oracle.spec_accept(prow, qrow, T, x, u) else 1, 2)[1]
    if thr > 0:
        assert oracle.spec_accept(prow, qrow, T, x, thr - 1)
    if thr < TWO64:
        assert not oracle.spec_accept(prow, qrow, T, x, thr)
    return thr


def test_spec_sampling_emits_p_exactly():
    """Speculative sampling's guarantee (Sec. 2): with x drawn from q, the
    emitted token -- x when accepted, else the residual draw -- follows p.
    For random tiny rows the law is computed exactly with fractions from the
    oracle's own behaviour (each x's accept threshold and the residual draw's
    boundaries, found by bisection over u) and equals P_j / Zp to within the
    uniform's resolution.  The thresholds are ceil(2^64 P_x Zq / (Q_x Zp))
    and the residual boundaries those of max(0, P_j Zq - Q_j Zp), both in big
    integers here; a token outside the vocabulary is always rejected."""
    rng = np.random.default_rng(38)
    for _ in range(30):
        V = int(rng.integers(2, 6))
        T = float(rng.choice([0.4, 1.0, 2.0]))
        prow = f32_to_bf16_bits(rng.normal(0, 1.5, V).astype(np.float32))
        qrow = f32_to_bf16_bits(rng.normal(0, 1.5, V).astype(np.float32))
        P, Zp = oracle.row_weights(prow, T)
        Q, Zq = oracle.row_weights(qrow, T)
        P, Q = [int(v) for v in P], [int(v) for v in Q]
        assert _accept_threshold(prow, qrow, T, V + 3) == 0
        U = _boundaries(lambda u: oracle.residual_row(prow, qrow, T, u), V)
        Rj = [max(0, P[j] * Zq - Q[j] * Zp) for j in range(V)]
        SR = sum(Rj)
        if SR > 0:
            S = np.cumsum(Rj, dtype=object).tolist()
            assert U == [0] + [_ceil_div(S[j - 1] * TWO64, SR) for j in range(1, V)] + [TWO64]
        res = [Fraction(U[j + 1] - U[j], TWO64) for j in range(V)]
        law = [Fraction(0)] * V
        for x in range(V):
            thr = _accept_threshold(prow, qrow, T, x)
            exp_thr = (min(TWO64, _ceil_div(TWO64 * P[x] * Zq, Q[x] * Zp)) if Q[x] > 0
                       else (TWO64 if P[x] > 0 else 0))
            assert thr == exp_thr
            a, qx = Fraction(thr, TWO64), Fraction(Q[x], Zq)
            law[x] += qx * a
            for j in range(V):
                law[j] += qx * (1 - a) * res[j]
        for j in range(V):
            assert abs(law[j] - Fraction(P[j], Zp)) <= Fraction(4 * V, TWO64), (j, law, P, Zp)


def test_spec_with_one_hot_q_is_the_one_hot_rule():
    """A draft row whose distribution is one-hot at x (its logits are x's
    +8, the rest -inf): x is accepted iff u < 2^64 p(x), and the residual is
    p without x -- the law of the one-hot rule."""
    rng = np.random.default_rng(39)
    for _ in range(20):
        V = int(rng.integers(2, 7))
        T = float(rng.choice([0.5, 1.0]))
        prow = f32_to_bf16_bits(rng.normal(0, 1, V).astype(np.float32))
        x = int(rng.integers(V))
        qrow = np.full(V, 0xFF80, np.uint16)
        qrow[x] = f32_to_bf16_bits(np.float32([8.0]))[0]
        P, Zp = oracle.row_weights(prow, T)
        assert _accept_threshold(prow, qrow, T, x) == _ceil_div(TWO64 * int(P[x]), Zp)
        if int(P[x]) < Zp:
            U = _boundaries(lambda u: oracle.residual_row(prow, qrow, T, u), V)
            rest = sum(int(P[j]) for j in range(V) if j != x)
            for j in range(V):
                share = Fraction(U[j + 1] - U[j], TWO64)
                want = Fraction(0) if j == x else Fraction(int(P[j]), rest)
                assert abs(share - want) <= Fraction(1, 2 ** 62)


def test_spec_chain_step():
    """oracle.step with draft logits: a neural chain is tested row by row with
    the accept uniforms and ends at the first rejection with the residual draw
    (else the bonus from the last row); a copy draft keeps the one-hot rule.
    Checked against the per-row functions, and the first emitted token's
    frequency over many seeded steps against softmax(l / T) of row 0."""
    rng = np.random.default_rng(40)
    for _ in range(60):
        B, R, V = 4, int(rng.integers(2, 7)), int(rng.integers(2, 9))
        k = R - 1
        tokens = rng.integers(0, 3, (B, 30)).astype(np.int32)
        lengths = rng.integers(1, 31, B).astype(np.int32)
        logits = f32_to_bf16_bits(rng.normal(0, 1, (B, R, V)).astype(np.float32))
        qlog = f32_to_bf16_bits(rng.normal(0, 1, (B, R, V)).astype(np.float32))
        un, ua = _u64(rng, (B, R)), _u64(rng, (B, R))
        ntok = rng.integers(-1, V + 1, (B, R)).astype(np.int32)
        nn = rng.integers(1, R + 1, B).astype(np.int32)
        T = float(rng.choice([0.3, 0.8, 1.5]))
        cfg = oracle.make_cfg((2, 1), 1, k, float(rng.choice([0.0, np.inf])))
        hid = np.zeros((B, 4), np.uint16)
        res = oracle.step(tokens, lengths, hid, np.zeros(4, np.float32), 0.0, ntok, None, nn,
                          logits, cfg, temperature=T, uniforms=un, draft_logits=qlog,
                          accept_uniforms=ua)
        for b in range(B):
            dn, dtok = int(res["dn"][b]), res["dtok"][b]
            if res["use_copy"][b]:
                am = [oracle.sample_row(logits[b, r], T, un[b, r]) if r < dn else -1
                      for r in range(R)]
                exp = brute.accept(dtok, res["dpar"][b], dn, am, R)
                assert (res["accept_len"][b], res["bonus"][b]) == (exp[0], exp[2])
                continue
            a = dn - 1
            for r in range(dn - 1):
                if not oracle.spec_accept(logits[b, r], qlog[b, r], T, dtok[r + 1], ua[b, r]):
                    a = r
                    break
            y = (oracle.residual_row(logits[b, a], qlog[b, a], T, un[b, a]) if a + 1 < dn
                 else oracle.sample_row(logits[b, a], T, un[b, a]))
            exp_out = [int(dtok[r + 1]) for r in range(a)] + [y] + [-1] * (R - a - 1)
            assert res["accept_len"][b] == a and res["accept_node"][b] == a
            assert res["bonus"][b] == y
            assert res["out_tokens"][b].tolist() == exp_out
            assert res["amax"][b].tolist() == exp_out
    # the first emitted token follows p at row 0, whatever q drafted
    n, V, T = 30000, 5, 0.9
    prow = f32_to_bf16_bits(rng.normal(0, 1, V).astype(np.float32))
    qrow = f32_to_bf16_bits(rng.normal(0, 1, V).astype(np.float32))
    q = _softmax64(qrow, T)
    logits = np.zeros((n, 2, V), np.uint16)
    logits[:, 0] = prow
    qlog = np.zeros((n, 2, V), np.uint16)
    qlog[:, 0] = qrow
    ntok = np.zeros((n, 2), np.int32)
    ntok[:, 1] = rng.choice(V, n, p=q)                   # drafted from q
    res = oracle.step(np.zeros((n, 4), np.int32), np.ones(n, np.int32),
                      np.zeros((n, 0), np.uint16), np.zeros(0, np.float32), 0.0, ntok, None,
                      np.full(n, 2, np.int32), logits, oracle.make_cfg((1,), 1, 1, np.inf),
                      threads=8, temperature=T, uniforms=_u64(rng, (n, 2)),
                      draft_logits=qlog, accept_uniforms=_u64(rng, (n, 2)))
    first = res["out_tokens"][:, 0]
    p = _softmax64(prow, T)
    freq = np.bincount(first, minlength=V) / n
    np.testing.assert_allclose(freq, p, atol=4 * np.sqrt(p.max() / n) + 1e-3)
