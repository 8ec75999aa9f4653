"""Pins of the copy-mode labels (Sec. 3.2, Problem Formulation): hand-derived
cases, an independent byte-string formulation on random tiny sequences, and
properties of the rule (monotone in n, planted spans, n = 1)."""
import json
import os

import numpy as np
import pytest

import oracle
from paper_2609_20186_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _cases():
    with open(os.path.join(GOLDEN, "label_cases.jsonl")) as f:
        return [json.loads(s) for s in f if s.strip()]


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c["why"][:40])
def test_golden_labels(case):
    x = np.array([case["x"]], np.int32)
    assert oracle.copy_labels(x, [x.shape[1]], case["n"])[0].tolist() == case["labels"]


def brute_labels(x, L, n):
    """Span formulation: for every span length m >= n and start s, the span is
    copy-mode if bytes.find finds its encoding at an aligned offset before s."""
    x = np.asarray(x[:L], "<i4")
    lab = np.zeros(L, np.uint8)
    hay = x.tobytes()
    for m in range(n, L + 1):
        for s in range(0, L - m + 1):
            pat = x[s:s + m].tobytes()
            pos = -1
            start = 0
            while True:
                i = hay.find(pat, start)
                if i < 0 or i // 4 >= s:
                    break
                if i % 4 == 0:
                    pos = i // 4
                    break
                start = i + 1
            if pos >= 0:
                lab[s:s + m] = 1
    return lab


def test_labels_equal_span_brute_force():
    rng = np.random.default_rng(50)
    for _ in range(300):
        Lmax = int(rng.integers(1, 30))
        L = int(rng.integers(0, Lmax + 1))
        n = int(rng.integers(1, 6))
        x = rng.integers(0, int(rng.choice([2, 3, 5])), (1, Lmax)).astype(np.int32)
        got = oracle.copy_labels(x, [L], n)[0]
        exp = np.zeros(Lmax, np.uint8)
        exp[:L] = brute_labels(x[0], L, n)
        np.testing.assert_array_equal(got, exp, err_msg=f"{x[0, :L].tolist()} n={n}")


def test_label_properties():
    rng = np.random.default_rng(51)
    for _ in range(100):
        L = int(rng.integers(2, 200))
        x = rng.integers(0, 6, (1, L)).astype(np.int32)
        prev = None
        for n in range(1, 8):
            lab = oracle.copy_labels(x, [L], n)[0]
            if prev is not None:
                assert np.all(lab <= prev)            # a longer threshold labels less
            prev = lab
        first = {}
        lab1 = oracle.copy_labels(x, [L], 1)[0]
        for j in range(L):
            assert lab1[j] == (int(x[0, j]) in first)
            first.setdefault(int(x[0, j]), j)


def test_planted_spans_are_labelled():
    """Every position of a span copied from earlier in a C2-shaped context
    (spans of 32..256 tokens) is copy-mode at n = 5; unrelated i.i.d. draws
    over a large vocabulary label nothing."""
    wl = W.WORKLOADS["C2"]
    rng = np.random.default_rng(52)
    x = rng.integers(0, 1 << 30, (1, 3000)).astype(np.int32)
    assert oracle.copy_labels(x, [3000], 5).sum() == 0
    src = int(rng.integers(0, 1000))
    x[0, 2000:2100] = x[0, src:src + 100]
    lab = oracle.copy_labels(x, [3000], 5)[0]
    assert lab[2000:2100].all() and lab[:2000].sum() == 0 and lab[2100:].sum() == 0
    d = W.generate(wl, batch=[0], logits=False)
    lab = oracle.copy_labels(d["tokens"], d["lengths"], 5)[0]
    assert 0.2 < lab.mean() < 0.5                     # about the 30% span share
