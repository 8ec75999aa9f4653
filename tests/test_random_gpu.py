"""GPU parity on seeded random configurations: batch, context and vocabulary
sizes, n-gram lengths, gate, threshold, candidate count, draft length, trees,
ragged lengths and special logits drawn at random, each run in every launch
mode (and at T > 0 where the rows allow it) against the oracle."""
import numpy as np
import pytest

from gpu_helpers import assert_match, gpu_stages, gpu_step, oracle_step, say, to_device, \
    with_temperature
from test_parity_gpu import AUTO, FUSED, SPLIT, custom_case, workspace_left_clean

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_20186_amd import binding  # noqa: F401  (fails loudly if not built)


def random_config(seed):
    """One configuration the C ABI accepts (1 + W k <= R, lengths strictly
    descending in 1..64), sized so that the oracle finishes in about a second."""
    rng = np.random.default_rng(10_000 + seed)
    W = int(rng.choice([1, 1, 1, 2, 3, 10, 16]))
    k = int(rng.integers(0, 21 if W == 1 else 8))
    R = 1 + W * k + int(rng.integers(0, 12))
    tree = bool(rng.random() < 0.4)
    B = int(rng.integers(1, 24))
    Lmax = int(rng.choice([int(rng.integers(2, 200)), int(rng.integers(200, 3000)),
                           int(rng.integers(3000, 9000))]))
    V = int(rng.choice([int(rng.integers(1, 64)), int(rng.integers(64, 5000)) * 8,
                        int(rng.integers(5000, 70000))]))
    while B * R * V > 6_000_000 and B > 1:
        B = max(1, B // 2)
    while B * R * V > 6_000_000:
        V = max(1, V // 2)
    n_len = int(rng.integers(1, 5))
    if rng.random() < 0.15:
        lens = tuple(sorted(rng.choice(np.arange(1, 65), n_len, replace=False).tolist(),
                            reverse=True))
    else:
        lens = tuple(sorted(rng.choice(np.arange(1, 7), min(n_len, 6), replace=False).tolist(),
                            reverse=True))
    vocab = int(rng.choice([2, 3, 8, 50, 1000]))
    return dict(seed=20_000 + seed, B=B, Lmax=Lmax, V=V, R=R, k=k, lens=lens,
                kappa=int(rng.integers(1, 4)),
                theta=float(rng.choice([-np.inf, -0.3, 0.0, 0.3, np.inf])),
                d=int(rng.choice([0, 1, 64, 1027])), tree=tree,
                vocab=vocab, ragged=bool(rng.random() < 0.7),
                specials=bool(rng.random() < 0.2), ties=bool(rng.random() < 0.3),
                neg=bool(rng.random() < 0.15), n_cand=W,
                # planted acceptance needs every drafted token to be a row index
                plant=bool(rng.random() < 0.5) and vocab <= V)


@pytest.mark.parametrize("seed", range(48))
def test_random_config_parity(seed):
    cfg = random_config(seed)
    say(f"[random] seed {seed}: " + ", ".join(f"{k}={v}" for k, v in cfg.items()))
    d = custom_case(**cfg)
    exp = oracle_step(d)
    dev = to_device(d)
    for mode in (AUTO, FUSED, SPLIT):
        got, ws = gpu_step(dev, d, mode)
        assert_match(got, exp, what=f"random {seed} mode {mode}")
        assert workspace_left_clean(ws, d)
    stages, _ = gpu_stages(dev, d)
    assert_match(stages, exp, what=f"random {seed} stages")
    if cfg["V"] % 8 == 0 and seed % 2 == 0:
        T = float(np.random.default_rng(seed).choice([0.2, 0.7, 1.5]))
        dt = with_temperature(d, T, seed=30_000 + seed)
        expt = oracle_step(dt)
        devt = to_device(dt)
        for mode in (AUTO, FUSED, SPLIT):
            got, ws = gpu_step(devt, dt, mode)
            assert_match(got, expt, what=f"random {seed} T={T} mode {mode}")
            assert workspace_left_clean(ws, dt)


MAX_CASES = {
    # the largest vocabulary the draw at T > 0 accepts, on the streamed path
    # (R > 64), with 16 copy candidates
    "max_vocab": dict(seed=90, B=2, Lmax=2000, V=524288, R=65, k=4, lens=(3, 2, 1), kappa=1,
                      theta=-0.2, vocab=20, n_cand=16, plant=True),
    # the most rows per sequence: 16 candidates of 63 tokens (1009 nodes) in
    # 1024 rows, accept walks over hundreds of nodes
    "max_rows": dict(seed=91, B=3, Lmax=3000, V=64, R=1024, k=63, lens=(3, 2, 1), kappa=1,
                     theta=-0.2, vocab=3, n_cand=16, plant=True),
}


@pytest.mark.parametrize("case", sorted(MAX_CASES))
def test_maximum_sizes(case):
    say(f"[max] {case}")
    d = custom_case(**MAX_CASES[case])
    for T in (0.0, 0.7):
        dt = with_temperature(d, T, seed=40_000) if T > 0 else d
        exp = oracle_step(dt)
        dev = to_device(dt)
        for mode in (AUTO, FUSED, SPLIT):
            got, ws = gpu_step(dev, dt, mode)
            assert_match(got, exp, what=f"{case} T={T} mode {mode}")
            assert workspace_left_clean(ws, dt)
