"""GPU parity of the draw at sampling temperature T > 0 (App. A) against the
oracle: every drawn token (amax) and every accept output bit-exact, the probe
logit within 1e-3.  The draws use seeded uniforms passed to both sides."""
import numpy as np
import pytest

from gpu_helpers import (assert_match, gpu_stages, gpu_step, oracle_step, planted_workload, say,
                         to_device, with_temperature)
from test_parity_gpu import SPLIT, FUSED, AUTO, custom_case, workspace_left_clean

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_20186_amd import binding  # noqa: F401


@pytest.mark.parametrize("name,T", [("C1", 0.7), ("C2", 0.2), ("C2", 0.7), ("C2", 1.5),
                                    ("C3", 1.0), ("C4", 0.7), ("C2W10", 0.7)])
def test_sampled_workload_parity(name, T):
    say(f"[sample] {name} T={T}")
    d = with_temperature(planted_workload(name), T, seed=100 + int(10 * T))
    exp = oracle_step(d)
    dev = to_device(d)
    got, ws = gpu_step(dev, d, AUTO)
    assert_match(got, exp, what=f"{name} T={T}")
    assert workspace_left_clean(ws, d)
    say(f"[sample] {name} T={T}: mean accept {exp['accept_len'].mean():.2f}")


def test_sampled_c5_full_size():
    """C5 at T = 0.7, full size: every sequence and every output against the
    oracle, in both launch modes, workspace left zeroed."""
    say("[sample] C5 T=0.7, all 256 sequences")
    d = with_temperature(planted_workload("C5"), 0.7, seed=105)
    exp = oracle_step(d)
    dev = to_device(d)
    for mode in (AUTO, FUSED):
        got, ws = gpu_step(dev, d, mode)
        assert_match(got, exp, what=f"C5 T=0.7 mode {mode}")
        assert workspace_left_clean(ws, d)
    say(f"[sample] C5 T=0.7: mean accept {exp['accept_len'].mean():.2f}")


SAMPLE_CASES = {
    "specials": dict(seed=60, B=4, Lmax=64, V=16, R=5, k=4, lens=(3, 1), kappa=1, theta=0.0,
                     vocab=4, specials=True),
    "ties": dict(seed=61, B=7, Lmax=300, V=8, R=6, k=5, lens=(4, 2), kappa=2, theta=-0.3,
                 vocab=3, ties=True),
    "tree30": dict(seed=62, B=9, Lmax=2000, V=304, R=30, k=7, lens=(3, 2, 1), kappa=1,
                   theta=0.0, vocab=3, tree=True, plant=True),
    # few enough rows (B * R <= the CU count) for the polled draw
    "tree30_polled": dict(seed=71, B=8, Lmax=1500, V=304, R=30, k=7, lens=(3, 2, 1), kappa=1,
                          theta=0.0, vocab=3, tree=True, plant=True),
    # polled draws over more than 64 (chunk, wave) entries per row (the
    # two-level search), up to the largest vocabulary
    "wide_vocab_polled": dict(seed=72, B=3, Lmax=300, V=200000, R=4, k=3, lens=(2, 1), kappa=1,
                              theta=0.0, vocab=10, plant=True),
    "max_vocab_polled": dict(seed=73, B=2, Lmax=200, V=524288, R=3, k=2, lens=(2, 1), kappa=1,
                             theta=-np.inf, vocab=10, plant=True),
    "tree100": dict(seed=63, B=4, Lmax=500, V=40, R=100, k=10, lens=(2, 1), kappa=1, theta=0.0,
                    vocab=2, tree=True, ties=True),
    "w10_d20": dict(seed=64, B=6, Lmax=3000, V=3000, R=204, k=20, lens=(3, 2, 1), kappa=1,
                    theta=-0.2, vocab=30, n_cand=10, plant=True),
    "multi_chunk_rows": dict(seed=65, B=3, Lmax=900, V=40000, R=4, k=3, lens=(2, 1), kappa=1,
                             theta=-np.inf, vocab=10, plant=True),
    "negative_rows": dict(seed=70, B=3, Lmax=200, V=40000, R=4, k=3, lens=(2, 1), kappa=1,
                          theta=0.0, vocab=10, neg=True),
    "v8": dict(seed=66, B=5, Lmax=40, V=8, R=3, k=2, lens=(1,), kappa=1, theta=0.0, vocab=3),
    # more than 256 sequences with long drafts: per-row weight sums (not the
    # streamed ones), then the accept epilogue over more than 64 nodes
    "tree70_wide_batch": dict(seed=69, B=260, Lmax=96, V=64, R=70, k=5, lens=(2, 1), kappa=1,
                              theta=0.0, vocab=3, tree=True, ties=True),
}


def test_sampled_dirty_sample_workspace():
    """The sample workspace needs no initialization: filled with 0xFF bytes
    before each call (the polled draw's sum slots included, which the row
    maxima launch clears), C2 at T = 0.7 still matches the oracle in every
    launch mode."""
    import torch
    from paper_2609_20186_amd import binding as sd
    say("[sample] C2 T=0.7, sample workspace of 0xFF bytes")
    d = with_temperature(planted_workload("C2"), 0.7, seed=106)
    exp = oracle_step(d)
    dev = to_device(d)
    B, R = d["ntok"].shape
    sws = sd.alloc_sample_workspace(B, R, d["logits"].shape[2])
    for mode in (AUTO, FUSED, SPLIT):
        sws.fill_(255)
        got, ws = gpu_step(dev, d, mode, sws=sws)
        assert_match(got, exp, what=f"C2 T=0.7 dirty sample workspace, mode {mode}")
        assert workspace_left_clean(ws, d)


@pytest.mark.parametrize("T", [1e-4, 0.5, 3.0, 1e6])
@pytest.mark.parametrize("case", sorted(SAMPLE_CASES))
def test_sampled_edge_case_parity(case, T):
    say(f"[sample-edge] {case} T={T}")
    d = with_temperature(custom_case(**SAMPLE_CASES[case]), T, seed=7 + len(case))
    exp = oracle_step(d)
    dev = to_device(d)
    for mode in (AUTO, FUSED, SPLIT):
        got, ws = gpu_step(dev, d, mode)
        assert_match(got, exp, what=f"{case} T={T} mode {mode}")
        assert workspace_left_clean(ws, d)
    stages, _ = gpu_stages(dev, d)
    assert_match(stages, exp, what=f"{case} T={T} stages")


def test_sampling_rejects_unsupported_rows():
    """V not a multiple of 8 (rows not 16-byte aligned) and T <= 0 are refused
    before any launch."""
    import torch
    from paper_2609_20186_amd import binding as sd
    d = custom_case(seed=67, B=2, Lmax=20, V=12, R=3, k=2, lens=(1,), kappa=1, theta=0.0,
                    vocab=3)
    d = with_temperature(d, 0.5, seed=1)
    dev = to_device(d)
    o = sd.alloc_outputs(2, 3, 2)
    with pytest.raises(sd.SwitchsdError) as e:
        sd.switchsd_verify_sample(dev["logits"], 0.5, dev["uniforms"], o["dtok"], o["dpar"],
                                  o["dn"], o["accept_len"], o["accept_node"], o["bonus"],
                                  o["out_tokens"], o["amax"], sd.alloc_workspace(2, 3),
                                  sd.alloc_sample_workspace(2, 3, 12))
    assert e.value.status == -1
    d2 = with_temperature(custom_case(seed=68, B=2, Lmax=20, V=16, R=3, k=2, lens=(1,), kappa=1,
                                      theta=0.0, vocab=3), 0.5, seed=2)
    dev2 = to_device(d2)
    for T in (0.0, -1.0, float("nan"), float("inf")):
        with pytest.raises(sd.SwitchsdError):
            sd.switchsd_verify_sample(dev2["logits"], T, dev2["uniforms"], o["dtok"],
                                      o["dpar"], o["dn"], o["accept_len"], o["accept_node"],
                                      o["bonus"], o["out_tokens"], o["amax"],
                                      sd.alloc_workspace(2, 3),
                                      sd.alloc_sample_workspace(2, 3, 16))
    torch.cuda.synchronize()
