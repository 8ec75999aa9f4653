"""The C ABI library loads, exports every declared entry point, and rejects bad
arguments on the host before any HIP call (no GPU needed: only invalid calls
are made here, which return before touching the device)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2609_20186_amd import binding as sd

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "switchsd.h")

OK, EINVAL, ESHAPE, EHIP, EWORKSPACE, EDEVICE, ESCRATCH = 0, -1, -2, -3, -4, -5, -6


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(switchsd_\w+)\s*\(", text, re.M)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert set(names) >= {"switchsd_ngram_match", "switchsd_probe_score",
                          "switchsd_select_draft", "switchsd_verify_accept",
                          "switchsd_tree_mask", "switchsd_step", "switchsd_workspace_bytes",
                          "switchsd_status_string"}
    assert set(names) == set(sd.EXPORTS)
    lib = ctypes.CDLL(sd.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings_and_workspace_size():
    for s in (OK, EINVAL, ESHAPE, EHIP, EWORKSPACE, EDEVICE, ESCRATCH):
        assert sd.status_string(s) and sd.status_string(s) != "unknown status"
    assert sd.status_string(17) == "unknown status"
    assert sd.workspace_bytes(32, 8) >= 32 * 8 * 8 + 32 * 8 * 4 + 2 * 32 * 4
    # per sequence: 3 lines, two key lines, a ticket line, and for R <= 64 the
    # fused step's per-segment row keys (R * 16 u64)
    assert sd.workspace_bytes(1, 8) == 3 * 256 + 2 * 256 + 256 + 8 * 16 * 8
    assert sd.workspace_bytes(1, 65) == 3 * 256 + 2 * 768 + 512
    assert sd.workspace_bytes(64, 8) >= sd.workspace_bytes(32, 8)
    assert sd.workspace_bytes(-1, 8) == 0
    assert sd.workspace_bytes(2, 8, -1, 0) == 0 and sd.workspace_bytes(2, 8, 16, -1) == 0
    # candidate lists only with several candidates over several scan tiles
    # (1024 positions each)
    assert sd.workspace_bytes(2, 8, 1024, 10) == sd.workspace_bytes(2, 8)
    # per-tile match slots (8 int32 per tile, whole lines) for 2..64 tiles
    assert sd.workspace_bytes(2, 8, 1025, 1) == sd.workspace_bytes(2, 8) + 2 * 256
    assert sd.workspace_bytes(2, 8, 64 * 1024, 1) == sd.workspace_bytes(2, 8) + 2 * 2 * 1024
    assert sd.workspace_bytes(2, 8, 64 * 1024 + 1, 1) == sd.workspace_bytes(2, 8)
    assert sd.workspace_bytes(2, 8, 1025, 10) > sd.workspace_bytes(2, 8)
    extra = sd.workspace_bytes(2, 8, 3 * 1024, 10) - sd.workspace_bytes(2, 8)
    assert extra >= 2 * 3 * 8 * 10 * 4 and extra % 256 == 0


# Host buffers stand in for device pointers: every call below fails validation
# and never reaches HIP.
_buf = np.zeros(1 << 16, np.uint8)
P = _buf.ctypes.data
WS = (P + 255) & ~255


def step_args(**kw):
    a = sd.StepArgs()
    for f, _ in sd.StepArgs._fields_:
        if f not in ("B", "Lmax", "d", "R", "V", "bias", "cfg", "mode", "temperature",
                     "uniforms", "sample_workspace", "sample_workspace_bytes", "commit",
                     "draft_pos", "lag", "draft_logits", "accept_uniforms"):
            setattr(a, f, P)
    a.B, a.Lmax, a.d, a.R, a.V = 2, 16, 8, 8, 100
    a.cfg = sd.make_cfg((3, 2, 1), 1, 7, 0.0)
    for k, v in kw.items():
        setattr(a, k, v)
    return a


def call_step(a, ws=WS, nbytes=4096):
    return sd.lib.switchsd_step(ctypes.byref(a), ws, nbytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(B=-1), ESHAPE), (dict(Lmax=0), ESHAPE), (dict(d=-1), ESHAPE), (dict(R=0), ESHAPE),
    (dict(R=2000), ESHAPE), (dict(V=0), ESHAPE), (dict(R=7), ESHAPE),   # k + 1 > R
    (dict(cfg=sd.make_cfg((3, 2, 1), 1, 7, 0.0, n_cand=2)), ESHAPE),     # 1 + 2 k > R
    (dict(mode=3), EINVAL), (dict(tokens=None), EINVAL), (dict(logits=None), EINVAL),
    (dict(logits=P + 1), EINVAL), (dict(out_tokens=None), EINVAL), (dict(dn=None), EINVAL),
    (dict(hidden=None), EINVAL), (dict(nn=None), EINVAL),
])
def test_step_rejects(kw, code):
    assert call_step(step_args(**kw)) == code


def test_step_optional_pointers_and_empty_batch():
    # B = 0 is a no-op even with every pointer null
    a = sd.StepArgs()
    a.B, a.Lmax, a.d, a.R, a.V = 0, 1, 0, 1, 1
    a.cfg = sd.make_cfg((1,), 1, 0, 0.0)
    assert call_step(a, ws=None, nbytes=0) == OK
    # d = 0 needs no hidden/w; k = 0 needs no copy_tokens (still rejected later
    # for the deliberately tiny workspace, before any HIP call)
    a = step_args(d=0, hidden=None, w=None)
    assert call_step(a, nbytes=16) == EWORKSPACE


@pytest.mark.parametrize("cfg", [
    dict(ngram_lens=(), kappa=1), dict(ngram_lens=(2, 3), kappa=1), dict(ngram_lens=(3, 3)),
    dict(ngram_lens=(65,)), dict(ngram_lens=(0,)), dict(ngram_lens=(3,), kappa=0),
    dict(ngram_lens=(3,), k=-1), dict(ngram_lens=(3,), n_cand=-1),
    dict(ngram_lens=(3,), n_cand=17),
])
def test_bad_cfg(cfg):
    c = sd.make_cfg(**{"kappa": 1, "k": 7, **cfg})
    if not cfg.get("ngram_lens"):
        c.n_ngram = 0
    assert call_step(step_args(cfg=c)) == EINVAL
    rc = sd.lib.switchsd_ngram_match(P, P, 2, 16, ctypes.byref(c), P, P, P, P, WS, 4096, None)
    assert rc == EINVAL


def test_workspace_checks():
    a = step_args()
    need = sd.workspace_bytes(2, 8)
    assert call_step(a, ws=None) == EWORKSPACE
    assert call_step(a, ws=WS + 8, nbytes=need) == EWORKSPACE       # misaligned
    assert call_step(a, ws=WS, nbytes=need - 1) == EWORKSPACE       # too small


def test_stage_entry_points_reject():
    cfg = sd.make_cfg((3, 2, 1), 1, 7, 0.0)
    lib = sd.lib
    assert lib.switchsd_ngram_match(P, P, -1, 16, ctypes.byref(cfg), P, P, P, P, WS, 4096,
                                    None) == ESHAPE
    assert lib.switchsd_ngram_match(None, P, 2, 16, ctypes.byref(cfg), P, P, P, P, WS, 4096,
                                    None) == EINVAL
    assert lib.switchsd_ngram_match(P, P, 0, 16, ctypes.byref(cfg), None, None, None, None,
                                    None, 0, None) == OK
    assert lib.switchsd_probe_score(P, P, 0.0, 2, -1, P, None) == ESHAPE
    assert lib.switchsd_probe_score(None, P, 0.0, 2, 8, P, None) == EINVAL
    assert lib.switchsd_probe_score(P, P, 0.0, 0, 8, None, None) == OK
    assert lib.switchsd_select_draft(P, P, P, P, P, P, P, 2, 7, ctypes.byref(cfg), P, P, P, P,
                                     None) == ESHAPE           # k + 1 > R
    assert lib.switchsd_select_draft(P, P, P, P, None, P, P, 2, 8, ctypes.byref(cfg), P, P, P,
                                     P, None) == EINVAL
    assert lib.switchsd_verify_accept(P, 2, 8, 0, P, P, P, P, P, P, P, P, WS, 4096,
                                      None) == ESHAPE
    assert lib.switchsd_verify_accept(P + 1, 2, 8, 100, P, P, P, P, P, P, P, P, WS, 4096,
                                      None) == EINVAL
    assert lib.switchsd_verify_accept(P, 2, 8, 100, P, P, P, P, P, P, P, P, WS, 8,
                                      None) == EWORKSPACE
    c2 = sd.make_cfg((3, 2, 1), 1, 7, 0.0, n_cand=3)
    assert lib.switchsd_select_draft(P, P, P, P, P, P, P, 2, 21, ctypes.byref(c2), P, P, P, P,
                                     None) == ESHAPE           # 1 + W k > R
    # a multi-candidate match over several tiles needs the candidate lists
    need1 = sd.workspace_bytes(2, 0, 3 * 2048, 1)
    assert lib.switchsd_ngram_match(P, P, 2, 3 * 2048, ctypes.byref(c2), P, P, P, P, WS, need1,
                                    None) == EWORKSPACE
    assert lib.switchsd_tree_mask(P, P, -1, 8, P, None) == ESHAPE
    assert lib.switchsd_tree_mask(P, P, 2, 0, P, None) == ESHAPE
    assert lib.switchsd_tree_mask(P, P, 2, 1025, P, None) == ESHAPE
    assert lib.switchsd_tree_mask(P, None, 2, 8, P, None) == EINVAL
    assert lib.switchsd_tree_mask(P, P, 2, 8, None, None) == EINVAL
    assert lib.switchsd_tree_mask(None, None, 0, 8, None, None) == OK


def test_sample_entry_point_rejects():
    lib = sd.lib
    A16 = (P + 15) & ~15
    SW = WS
    need = sd.sample_workspace_bytes(2, 8, 128)
    assert need % 256 == 0
    # 64-bit weight sums per 16 KB chunk and wave (4) for the p rows and for the
    # q rows; per block of 64 vectors of one row per sequence a residual and a
    # P sum (32 bytes); a test word and the two sums Zp, Zq per row
    assert sd.sample_workspace_bytes(2, 8, 128256) == 2 * (2 * 8 * 16 * 4 * 8) + \
        2 * 16 * 16 * 32 + 256 + 256
    assert sd.sample_workspace_bytes(-1, 8, 8) == 0

    def call(logits=A16, V=128, T=0.5, uni=P, sw=SW, swn=4096, ws=WS,
             wsn=sd.workspace_bytes(2, 8), q=None, ua=None, dpar=P):
        return lib.switchsd_verify_sample(logits, 2, 8, V, T, uni, q, ua, P, dpar, P, P, P, P,
                                          P, P, ws, wsn, sw, swn, None)
    for T in (0.0, -0.5, float("nan"), float("inf")):
        assert call(T=T) == EINVAL
    assert call(uni=None) == EINVAL
    assert call(V=100) == EINVAL                       # rows not 16-byte aligned
    assert call(logits=A16 + 2) == EINVAL
    assert call(V=64 * 8192 + 8) == ESHAPE             # more than 64 chunks per row
    assert call(sw=None) == EWORKSPACE
    assert call(sw=SW + 4) == EWORKSPACE
    assert call(swn=need - 1) == EWORKSPACE
    assert call(wsn=8) == EWORKSPACE
    # the draft's distribution: chains only, with its accept uniforms, aligned
    assert call(q=A16, ua=P, dpar=P) == EINVAL
    assert call(q=A16, ua=None, dpar=None) == EINVAL
    assert call(q=A16 + 2, ua=P, dpar=None) == EINVAL
    assert lib.switchsd_verify_sample(P, 0, 8, 128, 0.5, None, None, None, None, None, None,
                                      None, None, None, None, None, None, 0, None, 0,
                                      None) == OK
    a = step_args(temperature=0.7)                     # sampled step without uniforms
    a.uniforms = None
    assert call_step(a, nbytes=1 << 15) == EINVAL
    a = step_args(temperature=0.0, draft_logits=P, accept_uniforms=P)   # q needs T > 0
    assert call_step(a, nbytes=1 << 15) == EINVAL
    a = step_args(temperature=0.7, draft_logits=P, accept_uniforms=P)   # q needs chains
    assert call_step(a, nbytes=1 << 15) == EINVAL


def test_label_entry_point_rejects():
    lib = sd.lib
    need = sd.label_workspace_bytes(2, 100)
    # a window table per sequence: a power of two of at least 4 Lmax (and 64)
    # 32-bit slots
    assert need == 2 * 512 * 4
    assert sd.label_workspace_bytes(3, 4096) == 3 * 16384 * 4
    assert sd.label_workspace_bytes(1, 10) == 64 * 4
    assert sd.label_workspace_bytes(-1, 5) == 0 and sd.label_workspace_bytes(1, (1 << 28) + 1) == 0
    assert lib.switchsd_copy_labels(P, P, 1, (1 << 28) + 1, 5, P, WS, need, None) == ESHAPE
    assert lib.switchsd_copy_labels(P, P, -1, 100, 5, P, WS, need, None) == ESHAPE
    assert lib.switchsd_copy_labels(P, P, 2, 0, 5, P, WS, need, None) == ESHAPE
    assert lib.switchsd_copy_labels(P, P, 2, 100, 0, P, WS, need, None) == EINVAL
    assert lib.switchsd_copy_labels(P, P, 2, 100, 65, P, WS, need, None) == EINVAL
    assert lib.switchsd_copy_labels(P, None, 2, 100, 5, P, WS, need, None) == EINVAL
    assert lib.switchsd_copy_labels(P, P, 2, 100, 5, P, WS + 8, need, None) == EWORKSPACE
    assert lib.switchsd_copy_labels(P, P, 2, 4096, 5, P, WS, need, None) == EWORKSPACE
    assert lib.switchsd_copy_labels(None, None, 0, 100, 5, None, None, 0, None) == OK


def test_commit_entry_point_rejects():
    lib = sd.lib
    assert lib.switchsd_commit(P, P, -1, 16, P, 8, P, P, P, P, None) == ESHAPE
    assert lib.switchsd_commit(P, P, 2, 0, P, 8, P, P, P, P, None) == ESHAPE
    assert lib.switchsd_commit(P, P, 2, 16, P, 0, P, P, P, P, None) == ESHAPE
    assert lib.switchsd_commit(P, P, 2, 16, P, 8, P, P, None, P, None) == EINVAL
    assert lib.switchsd_commit(None, None, 0, 16, None, 8, None, None, None, None, None) == OK
    a = step_args(commit=1)                            # loop step without its counters
    assert call_step(a, nbytes=1 << 15) == EINVAL


def test_status_entry_point_rejects():
    lib = sd.lib
    need = sd.workspace_bytes(3, 0)
    assert lib.switchsd_workspace_status(WS, need, -1, P, None) == ESHAPE
    assert lib.switchsd_workspace_status(WS, need, 3, None, None) == EINVAL
    assert lib.switchsd_workspace_status(None, need, 3, P, None) == EWORKSPACE
    assert lib.switchsd_workspace_status(WS + 8, need, 3, P, None) == EWORKSPACE
    assert lib.switchsd_workspace_status(WS, need - 1, 3, P, None) == EWORKSPACE


def test_noalloc_entry_point_rejects():
    """Bad arguments and requests beyond the fixed scratch are refused on the
    host, before the first call's clear or any other HIP call."""
    lib = sd.lib
    assert lib.switchsd_step_noalloc(None, None) == EINVAL
    assert lib.switchsd_step_noalloc(ctypes.byref(step_args(B=-1)), None) == ESHAPE
    assert lib.switchsd_step_noalloc(ctypes.byref(step_args(tokens=None)), None) == EINVAL
    big = 32 * 2 ** 20 // sd.workspace_bytes(1, 8, 16) + 1
    assert sd.workspace_bytes(big, 8, 16) > 32 * 2 ** 20
    assert lib.switchsd_step_noalloc(ctypes.byref(step_args(B=big)), None) == ESCRATCH
    # the T > 0 scratch counts too
    a = step_args(B=512, R=64, V=128256, temperature=0.7, uniforms=P,
                  logits=(P + 15) & ~15)
    assert sd.workspace_bytes(512, 64, 16) < 32 * 2 ** 20
    assert sd.sample_workspace_bytes(512, 64, 128256) > 32 * 2 ** 20
    assert lib.switchsd_step_noalloc(ctypes.byref(a), None) == ESCRATCH
