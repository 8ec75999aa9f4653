"""Device-side failure reporting: the step's one bounded wait (the last scan
work-group of a sequence waiting for the probe work-group's flag) gives up
when a test knob makes the probe withhold its flag.  Every kernel still exits
normally; switchsd_workspace_status reports SWITCHSD_EDEVICE once and clears
it; the switch fell back to the neural draft; after the workspace is zeroed
again, the next step matches the oracle."""
import numpy as np
import pytest

from gpu_helpers import (assert_match, gpu_step, oracle_step, planted_workload, say, to_device,
                         with_temperature)
from test_parity_gpu import FUSED, SPLIT

pytestmark = pytest.mark.gpu

EDEVICE = -5


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_20186_amd import binding  # noqa: F401


@pytest.mark.parametrize("mode", [FUSED, SPLIT])
def test_probe_wait_give_up_is_reported(mode):
    import torch
    from paper_2609_20186_amd import binding as sd
    say(f"[errors] withheld probe flag, mode {mode}")
    d = planted_workload("C2")         # 4096-token contexts: 4 scan tiles + a probe work-group
    B, R = d["ntok"].shape
    dev = to_device(d)
    ws = sd.alloc_workspace(B, R, d["tokens"].shape[1])
    st = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    sd.switchsd_workspace_status(ws, B, st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    sd.withhold_probe_flag_for_tests(True)
    try:
        got, ws = gpu_step(dev, d, mode, ws=ws)
    finally:
        sd.withhold_probe_flag_for_tests(False)
    sd.switchsd_workspace_status(ws, B, st)
    torch.cuda.synchronize()
    assert int(st.item()) == EDEVICE
    assert not got["use_copy"].any()      # the switch fell back to the neural draft
    sd.switchsd_workspace_status(ws, B, st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0            # read and cleared
    ws.zero_()
    got, ws = gpu_step(dev, d, mode, ws=ws)
    assert_match(got, oracle_step(d), what=f"after give-up, mode {mode}")
    sd.switchsd_workspace_status(ws, B, st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    assert int(ws.count_nonzero()) == 0


def test_tile_poll_give_up_several_candidates():
    """With W = 10 copy candidates the scan tiles store their candidate lists
    before their slots; with sequence 0's first tile withheld the last tile's
    poll gives up, the status reports it, every other sequence still matches
    the oracle, the workspace is left zeroed once the status call has read the
    error, and the next step matches again."""
    import torch
    from paper_2609_20186_amd import binding as sd
    say("[errors] withheld scan tile, W = 10, split step")
    d = planted_workload("C2W10", batch=range(8))
    B, R = d["ntok"].shape
    dev = to_device(d)
    ws = sd.alloc_workspace(B, R, d["tokens"].shape[1], d["cfg"]["n_cand"])
    st = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    exp = oracle_step(d)
    sd.withhold_segment_for_tests(True)
    try:
        got, ws = gpu_step(dev, d, SPLIT, ws=ws)
    finally:
        sd.withhold_segment_for_tests(False)
    sd.switchsd_workspace_status(ws, B, st)
    torch.cuda.synchronize()
    assert int(st.item()) == EDEVICE
    rest = slice(1, None)
    assert_match(got, {k: v[rest] for k, v in exp.items()}, rows=rest,
                 what="other sequences while sequence 0's tile poll gave up")
    assert int(ws.count_nonzero()) == 0
    got, ws = gpu_step(dev, d, SPLIT, ws=ws)
    assert_match(got, exp, what="after the tile give-up")
    sd.switchsd_workspace_status(ws, B, st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    assert int(ws.count_nonzero()) == 0


def test_draw_poll_give_up_is_reported():
    """At T > 0 the row pollers of the draw wait for the rows' weight sums;
    with sequence 0's first sum work-group of row 0 withheld (and its first
    scan tile, whose poll gives up as well) the status reports it, every other
    sequence still matches the oracle, the workspace is left zeroed once the
    status call has read the error, and the next step matches again."""
    import torch
    from paper_2609_20186_amd import binding as sd
    say("[errors] withheld weight sums, fused step at T = 0.7")
    d = with_temperature(planted_workload("C2"), 0.7, seed=107)
    B, R = d["ntok"].shape
    dev = to_device(d)
    ws = sd.alloc_workspace(B, R, d["tokens"].shape[1])
    st = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    exp = oracle_step(d)
    sd.withhold_segment_for_tests(True)
    try:
        got, ws = gpu_step(dev, d, FUSED, ws=ws)
    finally:
        sd.withhold_segment_for_tests(False)
    sd.switchsd_workspace_status(ws, B, st)
    torch.cuda.synchronize()
    assert int(st.item()) == EDEVICE
    rest = slice(1, None)
    assert_match(got, {k: v[rest] for k, v in exp.items()}, rows=rest,
                 what="other sequences while sequence 0's draw gave up")
    assert int(ws.count_nonzero()) == 0
    got, ws = gpu_step(dev, d, FUSED, ws=ws)
    assert_match(got, exp, what="after the draw give-up")
    sd.switchsd_workspace_status(ws, B, st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    assert int(ws.count_nonzero()) == 0


def test_segment_poll_give_up_is_reported():
    """The fused step's accept epilogue polls the argmax segments' result
    slots, and the last of C2's four scan tiles polls the other tiles' match
    slots; with sequence 0's first segment of row 0 and its first tile
    withheld both polls give up, the status reports it, every other sequence
    still matches the oracle, and the workspace is left zeroed once the status
    call has read the error."""
    import torch
    from paper_2609_20186_amd import binding as sd
    say("[errors] withheld segment result, fused step")
    d = planted_workload("C2")
    B, R = d["ntok"].shape
    dev = to_device(d)
    ws = sd.alloc_workspace(B, R, d["tokens"].shape[1])
    st = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    exp = oracle_step(d)
    sd.withhold_segment_for_tests(True)
    try:
        got, ws = gpu_step(dev, d, FUSED, ws=ws)
    finally:
        sd.withhold_segment_for_tests(False)
    sd.switchsd_workspace_status(ws, B, st)
    torch.cuda.synchronize()
    assert int(st.item()) == EDEVICE
    rest = slice(1, None)
    assert_match(got, {k: v[rest] for k, v in exp.items()}, rows=rest,
                 what="other sequences while sequence 0 gave up")
    assert int(ws.count_nonzero()) == 0
    got, ws = gpu_step(dev, d, FUSED, ws=ws)
    assert_match(got, exp, what="after the segment give-up")
    sd.switchsd_workspace_status(ws, B, st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    assert int(ws.count_nonzero()) == 0
