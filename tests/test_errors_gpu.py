"""Device-side failure reporting: the step's one bounded wait (the last scan
work-group of a sequence waiting for the probe work-group's flag) gives up
when a test knob makes the probe withhold its flag.  Every kernel still exits
normally; switchsd_workspace_status reports SWITCHSD_EDEVICE once and clears
it; the switch fell back to the neural draft; after the workspace is zeroed
again, the next step matches the oracle."""
import numpy as np
import pytest

from gpu_helpers import assert_match, gpu_step, oracle_step, planted_workload, say, to_device
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
