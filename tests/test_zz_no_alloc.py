"""switchsd_step_noalloc (the library's own fixed device scratch instead of a
caller workspace) against switchsd_step with a caller workspace: every output
identical, on two calls in a row with the second one smaller, greedy and at
T = 0.7 (where the draw's scratch comes from the same array)."""
import numpy as np
import pytest

from gpu_helpers import oracle_step, planted_workload, say, sd_cfg, to_device, with_temperature

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_20186_amd import binding  # noqa: F401


def _both(d):
    """(outputs of switchsd_step with its own workspaces, outputs of
    switchsd_step_noalloc), each from fresh output tensors."""
    import torch
    from paper_2609_20186_amd import binding as sd
    dev = to_device(d)
    B, R = d["ntok"].shape
    V = d["logits"].shape[2]
    k, W = d["cfg"]["k"], d["cfg"].get("n_cand", 1)
    T = d.get("T", 0.0)
    res = []
    for noalloc in (False, True):
        out = sd.alloc_outputs(B, R, k, W)
        for t in out.values():
            t.fill_(-7)
        sws = sd.alloc_sample_workspace(B, R, V) if T > 0 and not noalloc else None
        args = sd.build_step_args(dev, out, sd_cfg(d), sd.MODE_AUTO, T, dev.get("uniforms"),
                                  sws if sws is not None else
                                  (torch.empty(256, dtype=torch.uint8, device="cuda")
                                   if T > 0 else None))
        if noalloc:
            sd.switchsd_step_noalloc(args)
        else:
            sd.switchsd_step(args, sd.alloc_workspace(B, R, d["tokens"].shape[1], W))
        torch.cuda.synchronize()
        res.append({key: v.cpu().numpy() for key, v in out.items()})
    return res


@pytest.mark.parametrize("T", [0.0, 0.7])
def test_noalloc_equals_step_two_calls(T):
    for i, name in enumerate(("C2", "C1")):        # the second call is smaller
        say(f"[noalloc] call {i + 1}: {name} T={T}")
        d = planted_workload(name)
        if T > 0:
            d = with_temperature(d, T, seed=500 + i)
        ref, got = _both(d)
        for key in ref:
            np.testing.assert_array_equal(got[key], ref[key], err_msg=f"{name} T={T} {key}")
        exp = oracle_step(d)
        for key in ("accept_len", "bonus", "out_tokens", "use_copy"):
            np.testing.assert_array_equal(got[key], exp[key], err_msg=f"{name} oracle {key}")
