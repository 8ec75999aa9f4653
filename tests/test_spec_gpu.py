"""GPU parity of speculative sampling with the draft's own distribution q
(Sec. 2; App. A at T > 0) against the oracle: accept tests, the residual draw
at the first rejection, the bonus draw, every output bit-exact and the
workspace left zeroed, in every launch mode of the step and through the stage
entry points.  The draft's tokens are drawn from q itself, as a draft model
would draw them."""
import numpy as np
import pytest

import brute
from gpu_helpers import (assert_match, gpu_stages, gpu_step, oracle_step, planted_workload, say,
                         to_device, with_temperature)
from paper_2609_20186_amd.workloads import f32_to_bf16_bits
from test_parity_gpu import AUTO, FUSED, SPLIT, custom_case, workspace_left_clean

pytestmark = pytest.mark.gpu

KINDS = ("same", "near", "far", "onehot", "near", "far")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_20186_amd import binding  # noqa: F401


def with_draft_distribution(d, T, seed, kinds=KINDS, invalid=False, degenerate=False):
    """Draft logits per sequence: equal to the target's ("same"), the target's
    plus N(0, 0.3) noise ("near"), independent N(0, 1) ("far") or one-hot at
    a random token ("onehot"); the neural draft's tokens are drawn from
    softmax(q / T) row by row.  invalid: some drafted tokens are -1 or V;
    degenerate: some q rows hold +inf or only NaN."""
    rng = np.random.default_rng(seed)
    d = dict(d)
    B, R, V = d["logits"].shape
    lf = brute.bf16_to_f32(d["logits"]).astype(np.float32)
    ql = np.empty_like(d["logits"])
    ntok = d["ntok"].copy()
    for b in range(B):
        kind = kinds[b % len(kinds)]
        if kind == "same":
            ql[b] = d["logits"][b]
        elif kind == "near":
            ql[b] = f32_to_bf16_bits((lf[b] + rng.normal(0, 0.3, (R, V))).astype(np.float32))
        elif kind == "far":
            ql[b] = f32_to_bf16_bits(np.clip(rng.normal(0, 1, (R, V)), -7.5, 7.5)
                                     .astype(np.float32))
        else:
            ql[b] = 0xFF80
            ql[b, np.arange(R), rng.integers(0, V, R)] = 0x4100          # 8.0
        qf = brute.bf16_to_f32(ql[b]).astype(np.float64)
        for r in range(R - 1):
            row = qf[r]
            ok = ~np.isnan(row)
            z = np.where(ok, (row - row[ok].max()) / T, -np.inf)
            pr = np.exp(z)
            ntok[b, r + 1] = int(rng.choice(V, p=pr / pr.sum()))
    if invalid:
        ntok[0, 1] = -1
        ntok[min(1, B - 1), min(2, R - 1)] = V
    if degenerate:
        ql[0, 0, 3] = 0x7F80                         # +inf: one-hot at the first +inf
        if B > 1:
            ql[1, 0, :] = 0x7FC0                     # all NaN: one-hot at index 0
    d["ntok"] = ntok
    d["draft_logits"] = ql
    d["accept_uniforms"] = rng.integers(0, 2 ** 64, (B, R), dtype=np.uint64)
    return d


def check_all_modes(d, what, stages=True):
    exp = oracle_step(d)
    dev = to_device(d)
    for mode in (AUTO, FUSED, SPLIT):
        got, ws = gpu_step(dev, d, mode)
        assert_match(got, exp, what=f"{what} mode {mode}")
        assert workspace_left_clean(ws, d), f"{what} mode {mode}: workspace not zeroed"
    if stages and not exp["use_copy"].any():
        got, _ = gpu_stages(dev, d)
        assert_match(got, exp, what=f"{what} stages")
    return exp


@pytest.mark.parametrize("name,T", [("C1", 0.7), ("C2", 0.7), ("C2", 0.2), ("C2", 1.5)])
def test_spec_workload_parity(name, T):
    say(f"[spec] {name} T={T}")
    d = with_draft_distribution(with_temperature(planted_workload(name), T, seed=300),
                                T, seed=301)
    exp = check_all_modes(d, f"{name} T={T}")
    neural = exp["use_copy"] == 0
    say(f"[spec] {name} T={T}: {int(neural.sum())} neural sequences, mean accept "
        f"{exp['accept_len'][neural].mean() if neural.any() else 0:.2f}")


def test_spec_neural_only_stages():
    """Every sequence neural (probe threshold +inf): the stage entry points
    verify every sequence with q and equal the step."""
    say("[spec] neural-only stages")
    d = planted_workload("C2")
    d["cfg"] = dict(d["cfg"], theta=np.inf)
    d = with_draft_distribution(with_temperature(d, 0.9, seed=302), 0.9, seed=303)
    exp = check_all_modes(d, "C2 neural-only")
    assert not exp["use_copy"].any()


SPEC_CASES = {
    "multi_chunk": dict(seed=80, B=6, Lmax=300, V=40000, R=5, k=4, lens=(2, 1), kappa=1,
                        theta=np.inf, vocab=10),
    "tiny_vocab_ties": dict(seed=81, B=7, Lmax=100, V=8, R=6, k=5, lens=(3, 1), kappa=1,
                            theta=np.inf, vocab=3, ties=True),
    "mixed_copy": dict(seed=82, B=9, Lmax=400, V=1024, R=7, k=6, lens=(3, 2, 1), kappa=1,
                       theta=0.0, vocab=4),
    "long_chain": dict(seed=83, B=7, Lmax=500, V=2048, R=100, k=10, lens=(2, 1), kappa=1,
                       theta=np.inf, vocab=30),
    "wide_batch": dict(seed=84, B=300, Lmax=64, V=256, R=4, k=3, lens=(1,), kappa=1,
                       theta=np.inf, vocab=50),
    # more than 256 blocks of 64 vectors per row: the residual draw finds the
    # chunk first, then the block
    "wide_vocab": dict(seed=88, B=3, Lmax=80, V=200000, R=4, k=3, lens=(2, 1), kappa=1,
                       theta=np.inf, vocab=8),
    # three copy candidates (the q row maxima in a launch of their own), copy
    # and neural drafts mixed
    "multi_candidate": dict(seed=91, B=6, Lmax=400, V=2048, R=12, k=3, lens=(2, 1), kappa=1,
                            theta=0.0, vocab=4, n_cand=3),
}


@pytest.mark.parametrize("T", [0.3, 1.0, 4.0])
@pytest.mark.parametrize("case", sorted(SPEC_CASES))
def test_spec_edge_case_parity(case, T):
    say(f"[spec-edge] {case} T={T}")
    d = with_temperature(custom_case(**SPEC_CASES[case]), T, seed=9 + len(case))
    d = with_draft_distribution(d, T, seed=10 + len(case), invalid=True, degenerate=True)
    check_all_modes(d, f"{case} T={T}")


def test_spec_residual_of_near_identical_distributions():
    """q equal to p except one far-tail element of row 0, one bf16 step lower
    in q: Zq is a few units below Zp, so at every other element the products
    P Zq and Q Zp lie within 2^-40 of each other (the residual launch compares
    them exactly) and its residual weight is 0.  With the accept uniform at
    its maximum, row 0's drafted token (another element) is rejected, and the
    residual draw must emit that tail element."""
    say("[spec] residual of near-identical distributions")
    T = 0.7
    B, R, V = 4, 4, 4096
    d = with_temperature(custom_case(seed=89, B=B, Lmax=50, V=V, R=R, k=3, lens=(1,),
                                     kappa=1, theta=np.inf, vocab=5), T, seed=90)
    d["nn"] = np.full(B, R, np.int32)
    lg = d["logits"].copy()
    ql = lg.copy()
    tails = []
    for b in range(B):
        x = int(d["ntok"][b, 1])
        j = (x + 1 + 97 * b) % V
        lg[b, 0, j] = 0xC140                         # -12.0: a small nonzero weight
        ql[b, 0, j] = 0xC141                         # -12.0625: one step lower in q
        tails.append(j)
    d["logits"] = lg
    d["draft_logits"] = ql
    d["accept_uniforms"] = np.full((B, R), 2 ** 64 - 1, np.uint64)
    exp = check_all_modes(d, "near-identical q")
    for b in range(B):
        assert exp["accept_len"][b] == 0
        assert exp["bonus"][b] == tails[b]


def test_spec_identical_distributions_accept_everything():
    """q = p: every valid drafted token is accepted (p(x)/q(x) = 1), and a
    drafted token outside the vocabulary is rejected with an empty residual,
    so the emitted token is drawn from p."""
    say("[spec] q = p")
    T = 0.8
    d = with_temperature(custom_case(seed=85, B=8, Lmax=50, V=4096, R=6, k=5, lens=(1,),
                                     kappa=1, theta=np.inf, vocab=5), T, seed=86)
    d["nn"] = np.full(8, 6, np.int32)
    d = with_draft_distribution(d, T, seed=87, kinds=("same",), invalid=True)
    exp = check_all_modes(d, "q = p")
    for b in range(2, 8):
        assert exp["accept_len"][b] == 5
    assert exp["accept_len"][0] == 0                 # ntok[0, 1] = -1 is rejected at row 0
