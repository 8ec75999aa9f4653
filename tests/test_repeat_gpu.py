"""Repeated back-to-back steps on one stream give identical results every time.

The step's work-groups hand results to each other through arrival tickets,
slots and flags in the workspace, whose order varies from launch to launch.
Each workload below runs many steps back to back (cycling over several output
sets, without synchronizing in between), then every output set must equal the
oracle's result and the workspace must be zero again."""
import numpy as np
import pytest

from gpu_helpers import (assert_match, oracle_step, planted_workload, say, sd_cfg, to_device,
                         with_temperature)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,T", [("C2", 0.0), ("C4", 0.0), ("C2W10", 0.0), ("C2", 0.7),
                                    ("C2W10", 0.7)])
def test_back_to_back_steps_agree(name, T):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_20186_amd import binding as sd
    say(f"[repeat] {name} T={T}")
    d = planted_workload(name, batch=list(range(8)))
    if T > 0:
        d = with_temperature(d, T, seed=91)
    exp = oracle_step(d)
    dev = to_device(d)
    B, R = dev["ntok"].shape
    k, W = d["cfg"]["k"], d["cfg"].get("n_cand", 1)
    ws = sd.alloc_workspace(B, R, dev["tokens"].shape[1], W)
    sws = sd.alloc_sample_workspace(B, R, dev["logits"].shape[2]) if T > 0 else None
    outs = [sd.alloc_outputs(B, R, k, W) for _ in range(4)]
    args = [sd.build_step_args(dev, o, sd_cfg(d), 0, T, dev.get("uniforms"), sws) for o in outs]
    for i in range(200):
        sd.switchsd_step(args[i % len(args)], ws)
    torch.cuda.synchronize()
    for j, o in enumerate(outs):
        got = {key: v.cpu().numpy() for key, v in o.items()}
        assert_match(got, exp, what=f"{name} T={T} output set {j}")
    assert int(ws.count_nonzero()) == 0 or W > 1   # W > 1 keeps its candidate lists
    if W > 1:
        need = sd.workspace_bytes(B, R)
        assert int(ws[:need].count_nonzero()) == 0
