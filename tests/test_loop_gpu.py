"""GPU decode loop (Sec. 3.3, KV Cache Synchronization): steps that append
their accepted tokens and bonus to the context and keep the draft model's
cache position and lag, against the oracle's loop; the stand-alone commit;
and the loop captured in a HIP graph and replayed."""
import numpy as np
import pytest

import oracle
from gpu_helpers import (ORACLE_THREADS, assert_match, ocfg, planted_workload, say, sd_cfg,
                         to_device, with_temperature)
from test_parity_gpu import AUTO, FUSED, SPLIT, custom_case
from test_spec_gpu import with_draft_distribution

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_20186_amd import binding  # noqa: F401


def widen(d, extra):
    """Room for `extra` more tokens per context."""
    d = dict(d)
    B, L = d["tokens"].shape
    t = np.zeros((B, L + extra), np.int32)
    t[:, :L] = d["tokens"]
    d["tokens"] = t
    return d


def oracle_loop(d, steps):
    c = d["cfg"]
    cfg = ocfg(c["lens"], c["kappa"], c["k"], c["theta"], c.get("n_cand", 1))
    tokens = d["tokens"].copy()
    lengths = np.clip(d["lengths"], 0, tokens.shape[1]).astype(np.int32)
    draft_pos = lengths.copy()
    T = d.get("T", 0.0)
    outs = []
    for s in range(steps):
        res = oracle.step(tokens, lengths, d["hidden"], d["w"], d["bias"], d["ntok"], d["npar"],
                          d["nn"], d["logits"], cfg, threads=ORACLE_THREADS, temperature=T,
                          uniforms=d["uniforms"] if T > 0 else None,
                          draft_logits=d.get("draft_logits"),
                          accept_uniforms=d.get("accept_uniforms"))
        lag = oracle.commit(tokens, lengths, draft_pos, res)
        outs.append(res)
    return outs, tokens, lengths, draft_pos, lag


class GpuLoop:
    def __init__(self, d, mode):
        import torch
        from paper_2609_20186_amd import binding as sd
        self.dev = to_device(d)
        B, R = d["ntok"].shape
        Lmax = d["tokens"].shape[1]
        c = d["cfg"]
        W = c.get("n_cand", 1)
        self.out = sd.alloc_outputs(B, R, c["k"], W)
        self.ws = sd.alloc_workspace(B, R, Lmax, W)
        self.dev["lengths"] = torch.from_numpy(
            np.clip(d["lengths"], 0, Lmax).astype(np.int32)).cuda()
        self.draft_pos = self.dev["lengths"].clone()
        self.lag = torch.zeros(B, dtype=torch.int32, device="cuda")
        T = d.get("T", 0.0)
        self.sws = sd.alloc_sample_workspace(B, R, d["logits"].shape[2]) if T > 0 else None
        self.args = sd.build_step_args(self.dev, self.out, sd_cfg(d), mode, T,
                                       self.dev.get("uniforms"), self.sws, self.draft_pos,
                                       self.lag, draft_logits=self.dev.get("draft_logits"),
                                       accept_uniforms=self.dev.get("accept_uniforms"))
        self.sd = sd

    def step(self):
        self.sd.switchsd_step(self.args, self.ws)

    def state(self):
        return (self.dev["tokens"].cpu().numpy(), self.dev["lengths"].cpu().numpy(),
                self.draft_pos.cpu().numpy(), self.lag.cpu().numpy())


LOOP_CASES = {
    "chain_fused": (dict(seed=80, B=5, Lmax=600, V=512, R=6, k=5, lens=(3, 2, 1), kappa=1,
                         theta=-0.3, vocab=6, plant=True), 0.0),
    "tree_split": (dict(seed=81, B=4, Lmax=700, V=304, R=30, k=7, lens=(3, 2, 1), kappa=1,
                        theta=0.0, vocab=4, tree=True, plant=True), 0.0),
    "w10_long": (dict(seed=82, B=3, Lmax=2500, V=1024, R=204, k=20, lens=(3, 2, 1), kappa=1,
                      theta=-0.2, vocab=20, n_cand=10, plant=True), 0.0),
    "chain_sampled": (dict(seed=83, B=5, Lmax=600, V=512, R=6, k=5, lens=(3, 2, 1), kappa=1,
                           theta=-0.3, vocab=6, plant=True), 0.6),
    # neural drafts verified with their distribution q: the residual launch
    # closes the step and commits
    "chain_sampled_q": (dict(seed=87, B=6, Lmax=600, V=512, R=6, k=5, lens=(3, 2, 1), kappa=1,
                             theta=-0.3, vocab=6), 0.6),
    "tiles_capacity": (dict(seed=84, B=3, Lmax=4200, V=256, R=9, k=8, lens=(3, 2, 1),
                            kappa=1, theta=-np.inf, vocab=5, ragged=False, plant=True), 0.0),
    # long drafts at T > 0: the streamed weight sums close the step and commit
    "w10_long_sampled": (dict(seed=85, B=3, Lmax=2500, V=1024, R=204, k=20, lens=(3, 2, 1),
                              kappa=1, theta=-0.2, vocab=20, n_cand=10, plant=True), 0.6),
    # more sequences than the streamed launches take: per-row sums with commit
    "wide_batch_sampled": (dict(seed=86, B=260, Lmax=96, V=64, R=70, k=5, lens=(2, 1),
                                kappa=1, theta=0.0, vocab=3, tree=True, plant=True), 0.6),
}


@pytest.mark.parametrize("case", sorted(LOOP_CASES))
def test_loop_parity(case):
    say(f"[loop] {case}")
    kw, T = LOOP_CASES[case]
    extra = 5 if case == "tiles_capacity" else 160          # the first runs into its capacity
    d = widen(custom_case(**kw), extra)
    if T > 0:
        d = with_temperature(d, T, seed=9)
    if case.endswith("_q"):
        d = with_draft_distribution(d, T, seed=10)
    steps = 12
    outs, t_exp, l_exp, dp_exp, lag_exp = oracle_loop(d, steps)
    for mode in (AUTO, FUSED, SPLIT):
        g = GpuLoop(d, mode)
        for s in range(steps):
            g.step()
            got = {k: v.cpu().numpy() for k, v in g.out.items()}
            assert_match(got, outs[s], what=f"{case} mode {mode} step {s}")
        t, l, dp, lag = g.state()
        np.testing.assert_array_equal(l, l_exp, err_msg=f"{case} lengths")
        np.testing.assert_array_equal(t, t_exp, err_msg=f"{case} tokens")
        np.testing.assert_array_equal(dp, dp_exp, err_msg=f"{case} draft_pos")
        np.testing.assert_array_equal(lag, lag_exp, err_msg=f"{case} lag")
    if case == "tiles_capacity":
        assert (l_exp == d["tokens"].shape[1]).all()          # every context filled up


def test_commit_entry_point_equals_step_commit():
    import torch
    from paper_2609_20186_amd import binding as sd
    say("[loop] stand-alone commit")
    d = widen(custom_case(**LOOP_CASES["tree_split"][0]), 50)
    outs, t_exp, l_exp, dp_exp, lag_exp = oracle_loop(d, 3)
    dev = to_device(d)
    B, R = d["ntok"].shape
    o = sd.alloc_outputs(B, R, d["cfg"]["k"])
    ws = sd.alloc_workspace(B, R, dev["tokens"].shape[1])
    dp = dev["lengths"].clone()
    lag = torch.zeros(B, dtype=torch.int32, device="cuda")
    args = sd.build_step_args(dev, o, sd_cfg(d))
    for s in range(3):
        sd.switchsd_step(args, ws)
        sd.switchsd_commit(dev["tokens"], dev["lengths"], o["out_tokens"], o["accept_len"],
                           o["use_copy"], dp, lag)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(dev["tokens"].cpu().numpy(), t_exp)
    np.testing.assert_array_equal(dev["lengths"].cpu().numpy(), l_exp)
    np.testing.assert_array_equal(dp.cpu().numpy(), dp_exp)
    np.testing.assert_array_equal(lag.cpu().numpy(), lag_exp)


@pytest.mark.parametrize("T,q", [(0.0, False), (0.6, False), (0.6, True)])
def test_loop_graph_replays(T, q):
    """Eight loop steps captured in one HIP graph; each replay starts from the
    initial state (restored by eager copies between replays) and must end in
    the eager loop's state."""
    import torch
    say(f"[loop] graph replays T={T} q={q}")
    d = widen(planted_workload("C2"), 8 * 8)
    if T > 0:
        d = with_temperature(d, T, seed=11)
    if q:
        d = with_draft_distribution(d, T, seed=12)
    g = GpuLoop(d, AUTO)
    t0, l0, dp0 = (g.dev["tokens"].clone(), g.dev["lengths"].clone(), g.draft_pos.clone())
    for _ in range(8):
        g.step()
    torch.cuda.synchronize()
    eager = g.state()

    def reset():
        g.dev["tokens"].copy_(t0)
        g.dev["lengths"].copy_(l0)
        g.draft_pos.copy_(dp0)
        torch.cuda.synchronize()

    reset()
    graph = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        g.step()                     # warm-up on the side stream before capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    reset()
    with torch.cuda.graph(graph):
        for _ in range(8):
            g.step()
    for rep in range(3):
        reset()
        graph.replay()
        torch.cuda.synchronize()
        got = g.state()
        for a, b, name in zip(got, eager, ("tokens", "lengths", "draft_pos", "lag")):
            np.testing.assert_array_equal(a, b, err_msg=f"replay {rep} {name}")
        _ = torch.ones(1024, device="cuda").sum().item()   # eager work between replays
