"""GPU copy-mode labels (Sec. 3.2) against the oracle, bit-exact."""
import numpy as np
import pytest

import oracle
from gpu_helpers import say
from paper_2609_20186_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_20186_amd import binding  # noqa: F401


def gpu_labels(tokens, lengths, n, ws=None):
    import torch
    from paper_2609_20186_amd import binding as sd
    B, Lmax = tokens.shape
    t = torch.from_numpy(np.ascontiguousarray(tokens, np.int32)).cuda()
    ln = torch.from_numpy(np.ascontiguousarray(lengths, np.int32)).cuda()
    lab = torch.full((B, Lmax), 7, dtype=torch.uint8, device="cuda")
    if ws is None:
        ws = torch.zeros(max(sd.label_workspace_bytes(B, Lmax), 256), dtype=torch.uint8,
                         device="cuda")
    sd.switchsd_copy_labels(t, ln, n, lab, ws)
    torch.cuda.synchronize()
    return lab.cpu().numpy(), ws


@pytest.mark.parametrize("n", [1, 2, 5, 8, 9, 64])
def test_labels_random_parity(n):
    """Small vocabularies (many repeats: windows sharing a table slot, and with
    vocabulary 1 a single content for every window), ragged and clamped
    lengths, contexts crossing the 256-position work-group boundaries, and
    windows longer than one 8-token read group (n = 9, 64)."""
    say(f"[labels] random n={n}")
    rng = np.random.default_rng(70 + n)
    for Lmax, vocab in ((1, 2), (63, 2), (64, 3), (65, 3), (300, 1), (700, 4), (1500, 20),
                        (2600, 2)):
        B = 5
        x = rng.integers(0, vocab, (B, Lmax)).astype(np.int32)
        if n == 64 and Lmax > 200:
            x[:, 150:] = x[:, :Lmax - 150]              # long repeats for the widest window
        lengths = rng.integers(0, Lmax + 1, B).astype(np.int32)
        lengths[0] = Lmax
        if B > 2:
            lengths[1], lengths[2] = 0, Lmax + 9
        got, ws = gpu_labels(x, lengths, n)
        exp = oracle.copy_labels(x, lengths, n)
        np.testing.assert_array_equal(got, exp, err_msg=f"Lmax={Lmax} vocab={vocab} n={n}")
        assert int(ws.count_nonzero()) == 0


@pytest.mark.parametrize("name,rows", [("C2", None), ("C4", [0, 5])])
def test_labels_workload_parity(name, rows):
    say(f"[labels] {name}")
    wl = W.WORKLOADS[name]
    d = W.generate(wl, logits=False)
    got, ws = gpu_labels(d["tokens"], d["lengths"], 5)
    idx = list(range(wl.B)) if rows is None else rows
    exp = oracle.copy_labels(d["tokens"][idx], d["lengths"][idx], 5)
    np.testing.assert_array_equal(got[idx], exp)
    assert int(ws.count_nonzero()) == 0
    say(f"[labels] {name}: copy-mode share {exp.mean():.3f}")
