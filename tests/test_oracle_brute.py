"""Pin the C oracle against the independent brute-force formulation.

Tiny random inputs (L <= 48, V in {2,3,5,8}) force many matches, overlapping
occurrences and argmax ties; logits are drawn from a handful of bf16 values
(including -0, +0, +-inf and NaN) and trees carry duplicate sibling tokens and
invalid parent links.  Every output of the oracle must equal the brute force.
"""
import numpy as np
import pytest

import brute
import oracle

BF16_VALUES = np.array([0xBF80, 0x8000, 0x0000, 0x3F80, 0x4000], np.uint16)  # -1,-0,0,1,2
BF16_SPECIAL = np.array([0x7F80, 0xFF80, 0x7FC0, 0xFFC0, 0x0001, 0x8001], np.uint16)  # +inf,-inf,NaN,-NaN,denormals


def random_case(rng, chain):
    B = int(rng.integers(1, 5))
    Lmax = int(rng.integers(1, 49))
    V = int(rng.choice([2, 3, 5, 8]))
    R = int(rng.integers(2, 9))
    k = int(rng.integers(0, R))                      # k + 1 <= R
    n_ng = int(rng.integers(1, 5))
    lens = sorted(rng.choice(np.arange(1, 9), n_ng, replace=False).tolist(), reverse=True)
    kappa = int(rng.integers(1, lens[0] + 2))
    theta = float(rng.choice([-np.inf, -0.75, 0.0, 0.5, np.inf]))
    d = int(rng.integers(0, 24))
    tokens = rng.integers(0, V, (B, Lmax)).astype(np.int32)
    lengths = rng.integers(0, Lmax + 1, B).astype(np.int32)
    if rng.random() < 0.2:
        lengths[0] = Lmax + 3                        # clamped to Lmax
    hidden = rng.choice(np.array([0x3F80, 0xBF80, 0x4040, 0x3E00, 0x0000], np.uint16), (B, d))
    w = rng.choice(np.array([0.25, -0.5, 1.0, 0.125, -0.375], np.float32), d)
    bias = float(rng.choice([0.0, -0.5, 0.25]))
    ntok = rng.integers(-1, V + 1, (B, R)).astype(np.int32)
    nn = rng.integers(0, R + 2, B).astype(np.int32)  # clamped to [1, R]
    if chain:
        npar = None
    else:
        npar = np.zeros((B, R), np.int32)
        for b in range(B):
            for i in range(R):
                npar[b, i] = -1 if i == 0 else int(rng.integers(0, i))
            if rng.random() < 0.3:
                i = int(rng.integers(1, R))
                npar[b, i] = int(rng.choice([-1, i, R + 2]))   # invalid: never accepted
    logits = rng.choice(BF16_VALUES, (B, R, V))
    if rng.random() < 0.3:
        m = rng.random((B, R, V)) < 0.2
        logits[m] = rng.choice(BF16_SPECIAL, int(m.sum()))
    return dict(tokens=tokens, lengths=lengths, hidden=hidden, w=w, bias=bias, ntok=ntok,
                npar=npar, nn=nn, logits=logits, lens=lens, kappa=kappa, k=k, theta=theta)


@pytest.mark.parametrize("chain", [True, False])
def test_oracle_equals_brute_force(chain):
    rng = np.random.default_rng(1234 + chain)
    for _ in range(400):
        c = random_case(rng, chain)
        cfg = oracle.make_cfg(c["lens"], c["kappa"], c["k"], c["theta"])
        got = oracle.step(c["tokens"], c["lengths"], c["hidden"], c["w"], c["bias"], c["ntok"],
                          c["npar"], c["nn"], c["logits"], cfg)
        exp = brute.step(c["tokens"], c["lengths"], c["hidden"], c["w"], c["bias"], c["ntok"],
                         c["npar"], c["nn"], c["logits"], c["lens"], c["kappa"], c["k"],
                         c["theta"])
        for key in exp:
            np.testing.assert_array_equal(got[key], exp[key], err_msg=f"{key} {c}")


@pytest.mark.parametrize("W", [2, 3, 10])
def test_oracle_equals_brute_force_multi_candidate(W):
    """W candidates (Sec. 3.3): the brute force collects every occurrence with
    repeated byte-string searches and builds the W chains itself."""
    rng = np.random.default_rng(4321 + W)
    for _ in range(300):
        c = random_case(rng, chain=True)
        k = int(rng.integers(0, 5))
        R = 1 + W * k + int(rng.integers(0, 3))
        c["ntok"] = rng.integers(-1, 4, (c["ntok"].shape[0], R)).astype(np.int32)
        c["logits"] = rng.choice(BF16_VALUES, (c["ntok"].shape[0], R, c["logits"].shape[2]))
        cfg = oracle.make_cfg(c["lens"], c["kappa"], k, c["theta"], n_cand=W)
        got = oracle.step(c["tokens"], c["lengths"], c["hidden"], c["w"], c["bias"], c["ntok"],
                          None, c["nn"], c["logits"], cfg)
        exp = brute.step(c["tokens"], c["lengths"], c["hidden"], c["w"], c["bias"], c["ntok"],
                         None, c["nn"], c["logits"], c["lens"], c["kappa"], k, c["theta"],
                         n_cand=W)
        for key in exp:
            np.testing.assert_array_equal(got[key], exp[key], err_msg=f"{key} W={W}")


def test_oracle_threads_do_not_change_results():
    rng = np.random.default_rng(7)
    c = random_case(rng, False)
    while c["tokens"].shape[0] < 3:
        c = random_case(rng, False)
    cfg = oracle.make_cfg(c["lens"], c["kappa"], c["k"], c["theta"])
    args = (c["tokens"], c["lengths"], c["hidden"], c["w"], c["bias"], c["ntok"], c["npar"],
            c["nn"], c["logits"], cfg)
    a = oracle.step(*args, threads=1)
    b = oracle.step(*args, threads=3)
    for key in a:
        np.testing.assert_array_equal(a[key], b[key])


def test_argmax_brute_on_wide_random_rows():
    """Wide rows of N(0,1) rounded to bf16: numpy's first-occurrence argmax of
    the exact float32 upcast is the definition (no NaN present)."""
    rng = np.random.default_rng(11)
    from paper_2609_20186_amd.workloads import f32_to_bf16_bits
    for V in (1, 7, 1000, 32000, 128256):
        row = f32_to_bf16_bits(rng.standard_normal(V).astype(np.float32))
        assert oracle.argmax_row(row) == int(np.argmax(brute.bf16_to_f32(row)))


def test_probe_matches_fsum_on_full_width():
    """The oracle's long-double sum, rounded once to float, equals the
    correctly rounded double sum (math.fsum) rounded to float, up to 1 ulp."""
    rng = np.random.default_rng(5)
    from paper_2609_20186_amd.workloads import f32_to_bf16_bits
    exact = 0
    for d in (1, 17, 1024, 4096, 8192):
        for _ in range(20):
            h = f32_to_bf16_bits(rng.standard_normal(d).astype(np.float32))
            w = (rng.standard_normal(d) / np.sqrt(d)).astype(np.float32)
            z1 = oracle.probe(h, w, -0.25)
            z2 = brute.probe(h, w, -0.25)
            assert abs(float(z1) - float(z2)) <= float(np.spacing(np.float32(abs(z2))))
            exact += int(z1 == z2)
    assert exact >= 98
