"""ctypes binding of libswitchsd.so (the C ABI in include/switchsd.h).

Argument marshalling only: every step runs in the HIP kernels of the library.
Tensors must be contiguous device tensors of the documented dtypes; bf16
arrays may be passed as torch.bfloat16 or as their 16-bit patterns
(int16/uint16).  Calls are asynchronous on the given (default: current) stream.
If the library is not built, importing raises instead of falling back to
anything else.
"""
import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libswitchsd.so")

MAX_NGRAM = 8
MAX_CAND = 16
MODE_AUTO, MODE_FUSED, MODE_SPLIT = 0, 1, 2

STATUS = {0: "OK", -1: "EINVAL", -2: "ESHAPE", -3: "EHIP", -4: "EWORKSPACE", -5: "EDEVICE",
          -6: "ESCRATCH"}

EXPORTS = ("switchsd_ngram_match", "switchsd_probe_score", "switchsd_select_draft",
           "switchsd_verify_accept", "switchsd_verify_sample", "switchsd_tree_mask",
           "switchsd_commit", "switchsd_step", "switchsd_copy_labels",
           "switchsd_workspace_bytes", "switchsd_sample_workspace_bytes",
           "switchsd_label_workspace_bytes", "switchsd_workspace_status", "switchsd_step_noalloc",
           "switchsd_test_withhold_probe_flag", "switchsd_test_withhold_segment",
           "switchsd_status_string")


class SwitchsdError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__(f"{fn} returned {status} ({STATUS.get(status, '?')}): "
                         f"{status_string(status)}")


class Cfg(ctypes.Structure):
    _fields_ = [("n_ngram", ctypes.c_int32),
                ("ngram_lens", ctypes.c_int32 * MAX_NGRAM),
                ("kappa", ctypes.c_int32),
                ("k", ctypes.c_int32),
                ("theta", ctypes.c_float),
                ("n_cand", ctypes.c_int32)]


def make_cfg(ngram_lens=(3, 2, 1), kappa=1, k=7, theta=0.0, n_cand=1):
    c = Cfg()
    c.n_ngram = len(ngram_lens)
    for i, n in enumerate(ngram_lens):
        c.ngram_lens[i] = int(n)
    c.kappa = int(kappa)
    c.k = int(k)
    c.theta = float(theta)
    c.n_cand = int(n_cand)
    return c


_P = ctypes.c_void_p
_I = ctypes.c_int32


class StepArgs(ctypes.Structure):
    _fields_ = [("tokens", _P), ("lengths", _P), ("hidden", _P), ("w", _P), ("ntok", _P),
                ("npar", _P), ("nn", _P), ("logits", _P),
                ("B", _I), ("Lmax", _I), ("d", _I), ("R", _I), ("V", _I),
                ("bias", ctypes.c_float), ("cfg", Cfg), ("mode", _I),
                ("match_n", _P), ("match_end", _P), ("copy_len", _P), ("copy_tokens", _P),
                ("z", _P), ("use_copy", _P), ("dtok", _P), ("dpar", _P), ("dn", _P),
                ("amax", _P), ("accept_len", _P), ("accept_node", _P), ("bonus", _P),
                ("out_tokens", _P), ("temperature", ctypes.c_float), ("uniforms", _P),
                ("sample_workspace", _P), ("sample_workspace_bytes", ctypes.c_size_t),
                ("commit", _I), ("draft_pos", _P), ("lag", _P),
                ("draft_logits", _P), ("accept_uniforms", _P)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2609_20186_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    S = ctypes.c_size_t
    lib.switchsd_ngram_match.argtypes = [_P, _P, _I, _I, ctypes.POINTER(Cfg), _P, _P, _P, _P,
                                         _P, S, _P]
    lib.switchsd_probe_score.argtypes = [_P, _P, ctypes.c_float, _I, _I, _P, _P]
    lib.switchsd_select_draft.argtypes = [_P, _P, _P, _P, _P, _P, _P, _I, _I,
                                          ctypes.POINTER(Cfg), _P, _P, _P, _P, _P]
    lib.switchsd_verify_accept.argtypes = [_P, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                           S, _P]
    lib.switchsd_tree_mask.argtypes = [_P, _P, _I, _I, _P, _P]
    lib.switchsd_verify_sample.argtypes = [_P, _I, _I, _I, ctypes.c_float, _P, _P, _P, _P, _P,
                                           _P, _P, _P, _P, _P, _P, _P, S, _P, S, _P]
    lib.switchsd_sample_workspace_bytes.argtypes = [_I, _I, _I]
    lib.switchsd_commit.argtypes = [_P, _P, _I, _I, _P, _I, _P, _P, _P, _P, _P]
    lib.switchsd_copy_labels.argtypes = [_P, _P, _I, _I, _I, _P, _P, S, _P]
    lib.switchsd_label_workspace_bytes.argtypes = [_I, _I]
    lib.switchsd_label_workspace_bytes.restype = S
    lib.switchsd_sample_workspace_bytes.restype = S
    lib.switchsd_step.argtypes = [ctypes.POINTER(StepArgs), _P, S, _P]
    lib.switchsd_step_noalloc.argtypes = [ctypes.POINTER(StepArgs), _P]
    lib.switchsd_workspace_bytes.argtypes = [_I, _I, _I, _I]
    lib.switchsd_workspace_bytes.restype = S
    lib.switchsd_workspace_status.argtypes = [_P, S, _I, _P, _P]
    for knob in ("switchsd_test_withhold_probe_flag", "switchsd_test_withhold_segment"):
        getattr(lib, knob).argtypes = [_I]
        getattr(lib, knob).restype = None
    lib.switchsd_status_string.argtypes = [ctypes.c_int]
    lib.switchsd_status_string.restype = ctypes.c_char_p
    for name in EXPORTS:
        if not name.startswith("switchsd_test_"):
            getattr(lib, name).restype = getattr(lib, name).restype or ctypes.c_int
    return lib


lib = _load()


def status_string(status):
    return lib.switchsd_status_string(int(status)).decode()


def workspace_bytes(B, R, Lmax=0, n_cand=0):
    return int(lib.switchsd_workspace_bytes(int(B), int(R), int(Lmax), int(n_cand)))


def sample_workspace_bytes(B, R, V):
    return int(lib.switchsd_sample_workspace_bytes(int(B), int(R), int(V)))


_DT = {"i32": (torch.int32,), "f32": (torch.float32,),
       "bf16": (torch.bfloat16, torch.int16, torch.uint16), "u8": (torch.uint8,),
       "u32": (torch.int32, torch.uint32), "u64": (torch.int64, torch.uint64)}


def _ptr(t, kind, name, optional=False):
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype not in _DT[kind]:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {_DT[kind]}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _check(fn, rc):
    if rc != 0:
        raise SwitchsdError(fn, rc)


def switchsd_ngram_match(tokens, lengths, cfg, match_n, match_end, copy_len, copy_tokens,
                         workspace, stream=None):
    B, Lmax = tokens.shape
    _check("switchsd_ngram_match", lib.switchsd_ngram_match(
        _ptr(tokens, "i32", "tokens"), _ptr(lengths, "i32", "lengths"), B, Lmax,
        ctypes.byref(cfg), _ptr(match_n, "i32", "match_n"), _ptr(match_end, "i32", "match_end"),
        _ptr(copy_len, "i32", "copy_len"), _ptr(copy_tokens, "i32", "copy_tokens", True),
        _ptr(workspace, "u8", "workspace"), workspace.numel(), _stream(stream)))


def switchsd_probe_score(hidden, w, bias, z, stream=None):
    B, d = hidden.shape
    _check("switchsd_probe_score", lib.switchsd_probe_score(
        _ptr(hidden, "bf16", "hidden"), _ptr(w, "f32", "w"), float(bias), B, d,
        _ptr(z, "f32", "z"), _stream(stream)))


def switchsd_select_draft(match_n, copy_len, copy_tokens, z, ntok, npar, nn, cfg, use_copy,
                          dtok, dpar, dn, stream=None):
    B, R = ntok.shape
    _check("switchsd_select_draft", lib.switchsd_select_draft(
        _ptr(match_n, "i32", "match_n"), _ptr(copy_len, "i32", "copy_len"),
        _ptr(copy_tokens, "i32", "copy_tokens", True), _ptr(z, "f32", "z"),
        _ptr(ntok, "i32", "ntok"), _ptr(npar, "i32", "npar", True), _ptr(nn, "i32", "nn"),
        B, R, ctypes.byref(cfg), _ptr(use_copy, "i32", "use_copy"), _ptr(dtok, "i32", "dtok"),
        _ptr(dpar, "i32", "dpar"), _ptr(dn, "i32", "dn"), _stream(stream)))


def switchsd_verify_accept(logits, dtok, dpar, dn, accept_len, accept_node, bonus, out_tokens,
                           amax, workspace, stream=None):
    B, R, V = logits.shape
    _check("switchsd_verify_accept", lib.switchsd_verify_accept(
        _ptr(logits, "bf16", "logits"), B, R, V, _ptr(dtok, "i32", "dtok"),
        _ptr(dpar, "i32", "dpar", True), _ptr(dn, "i32", "dn"),
        _ptr(accept_len, "i32", "accept_len"), _ptr(accept_node, "i32", "accept_node"),
        _ptr(bonus, "i32", "bonus"), _ptr(out_tokens, "i32", "out_tokens"),
        _ptr(amax, "i32", "amax", True), _ptr(workspace, "u8", "workspace"),
        workspace.numel(), _stream(stream)))


def switchsd_verify_sample(logits, temperature, uniforms, dtok, dpar, dn, accept_len,
                           accept_node, bonus, out_tokens, amax, workspace, sample_workspace,
                           stream=None, draft_logits=None, accept_uniforms=None):
    """uniforms, accept_uniforms: uint64 (or int64 holding the same bits) [B, R];
    draft_logits (bf16 [B, R, V]) verifies chains by speculative sampling with
    the draft's distribution."""
    B, R, V = logits.shape
    _check("switchsd_verify_sample", lib.switchsd_verify_sample(
        _ptr(logits, "bf16", "logits"), B, R, V, float(temperature),
        _ptr(uniforms, "u64", "uniforms"), _ptr(draft_logits, "bf16", "draft_logits", True),
        _ptr(accept_uniforms, "u64", "accept_uniforms", True), _ptr(dtok, "i32", "dtok"),
        _ptr(dpar, "i32", "dpar", True), _ptr(dn, "i32", "dn"),
        _ptr(accept_len, "i32", "accept_len"), _ptr(accept_node, "i32", "accept_node"),
        _ptr(bonus, "i32", "bonus"), _ptr(out_tokens, "i32", "out_tokens"),
        _ptr(amax, "i32", "amax", True), _ptr(workspace, "u8", "workspace"),
        workspace.numel(), _ptr(sample_workspace, "u8", "sample_workspace"),
        sample_workspace.numel(), _stream(stream)))


def switchsd_commit(tokens, lengths, out_tokens, accept_len, use_copy, draft_pos, lag,
                    stream=None):
    B, Lmax = tokens.shape
    R = out_tokens.shape[1]
    _check("switchsd_commit", lib.switchsd_commit(
        _ptr(tokens, "i32", "tokens"), _ptr(lengths, "i32", "lengths"), B, Lmax,
        _ptr(out_tokens, "i32", "out_tokens"), R, _ptr(accept_len, "i32", "accept_len"),
        _ptr(use_copy, "i32", "use_copy"), _ptr(draft_pos, "i32", "draft_pos"),
        _ptr(lag, "i32", "lag"), _stream(stream)))


def label_workspace_bytes(B, Lmax):
    return int(lib.switchsd_label_workspace_bytes(int(B), int(Lmax)))


def switchsd_copy_labels(tokens, lengths, n, labels, workspace, stream=None):
    """labels: uint8 [B, Lmax]; workspace: zeroed uint8 of label_workspace_bytes."""
    B, Lmax = tokens.shape
    _check("switchsd_copy_labels", lib.switchsd_copy_labels(
        _ptr(tokens, "i32", "tokens"), _ptr(lengths, "i32", "lengths"), B, Lmax, int(n),
        _ptr(labels, "u8", "labels"), _ptr(workspace, "u8", "workspace"), workspace.numel(),
        _stream(stream)))


def switchsd_workspace_status(workspace, B, status, stream=None):
    """Writes OK (0) or EDEVICE (-5) to the device int32 ``status`` [1] and
    clears the workspace's error words of B sequences."""
    _check("switchsd_workspace_status", lib.switchsd_workspace_status(
        _ptr(workspace, "u8", "workspace"), workspace.numel(), int(B),
        _ptr(status, "i32", "status"), _stream(stream)))


def withhold_probe_flag_for_tests(on):
    """Test support: force the step's bounded wait for the probe flag to give up."""
    lib.switchsd_test_withhold_probe_flag(1 if on else 0)


def withhold_segment_for_tests(on):
    """Test support: force the fused step's poll of the segment results to give up."""
    lib.switchsd_test_withhold_segment(1 if on else 0)


def switchsd_tree_mask(dpar, dn, mask, stream=None):
    """mask: uint32 (or int32 holding the same bits) [B, R, (R + 31) // 32]."""
    B, R = mask.shape[0], mask.shape[1]
    if mask.shape[2] != (R + 31) // 32:
        raise ValueError("mask must be [B, R, (R + 31) // 32]")
    _check("switchsd_tree_mask", lib.switchsd_tree_mask(
        _ptr(dpar, "i32", "dpar", True), _ptr(dn, "i32", "dn"), B, R,
        _ptr(mask, "u32", "mask"), _stream(stream)))


OUTPUTS = ("match_n", "match_end", "copy_len", "copy_tokens", "z", "use_copy", "dtok", "dpar",
           "dn", "amax", "accept_len", "accept_node", "bonus", "out_tokens")


def alloc_outputs(B, R, k, n_cand=1, device="cuda"):
    """Output tensors of a step; with n_cand > 1 the candidate outputs carry a
    W axis (match_end, copy_len [B, W], copy_tokens [B, W, k])."""
    i32 = dict(dtype=torch.int32, device=device)
    wsh = (B,) if n_cand <= 1 else (B, n_cand)
    return {"match_n": torch.empty(B, **i32), "match_end": torch.empty(wsh, **i32),
            "copy_len": torch.empty(wsh, **i32), "copy_tokens": torch.empty(wsh + (k,), **i32),
            "z": torch.empty(B, dtype=torch.float32, device=device),
            "use_copy": torch.empty(B, **i32), "dtok": torch.empty((B, R), **i32),
            "dpar": torch.empty((B, R), **i32), "dn": torch.empty(B, **i32),
            "amax": torch.empty((B, R), **i32), "accept_len": torch.empty(B, **i32),
            "accept_node": torch.empty(B, **i32), "bonus": torch.empty(B, **i32),
            "out_tokens": torch.empty((B, R), **i32)}


def alloc_sample_workspace(B, R, V, device="cuda"):
    return torch.empty(max(sample_workspace_bytes(B, R, V), 256), dtype=torch.uint8,
                       device=device)


def alloc_workspace(B, R, Lmax=0, n_cand=0, device="cuda"):
    """Zeroed once here; the kernels keep it usable for every later call."""
    return torch.zeros(max(workspace_bytes(B, R, Lmax, n_cand), 256), dtype=torch.uint8,
                       device=device)


def build_step_args(inp, out, cfg, mode=MODE_AUTO, temperature=0.0, uniforms=None,
                    sample_workspace=None, draft_pos=None, lag=None, draft_logits=None,
                    accept_uniforms=None):
    """StepArgs for switchsd_step.  ``inp`` holds device tensors tokens [B,Lmax],
    lengths [B], hidden [B,d], w [d], ntok [B,R], npar [B,R] or None, nn [B],
    logits [B,R,V] and the float ``bias``; ``out`` is from alloc_outputs.
    temperature > 0 draws the rows' tokens with ``uniforms`` [B,R] (uint64
    bits) and ``sample_workspace`` (alloc_sample_workspace); with
    ``draft_logits`` [B,R,V] and ``accept_uniforms`` [B,R] a chosen neural draft
    is verified by speculative sampling with its distribution.  With ``draft_pos``
    and ``lag`` [B] the step also commits (decode loop): tokens and lengths are
    then updated in place."""
    tokens, logits, hidden = inp["tokens"], inp["logits"], inp["hidden"]
    B, Lmax = tokens.shape
    R, V = logits.shape[1], logits.shape[2]
    a = StepArgs()
    a.tokens = _ptr(tokens, "i32", "tokens")
    a.lengths = _ptr(inp["lengths"], "i32", "lengths")
    a.hidden = _ptr(hidden, "bf16", "hidden")
    a.w = _ptr(inp["w"], "f32", "w")
    a.ntok = _ptr(inp["ntok"], "i32", "ntok")
    a.npar = _ptr(inp.get("npar"), "i32", "npar", True)
    a.nn = _ptr(inp["nn"], "i32", "nn")
    a.logits = _ptr(logits, "bf16", "logits")
    a.B, a.Lmax, a.d, a.R, a.V = B, Lmax, hidden.shape[1], R, V
    a.bias = float(inp["bias"])
    a.cfg = cfg
    a.mode = int(mode)
    for name in OUTPUTS:
        setattr(a, name, _ptr(out[name], "f32" if name == "z" else "i32", name,
                              optional=(name == "amax" or name == "copy_tokens")))
    if draft_pos is not None:
        a.commit = 1
        a.draft_pos = _ptr(draft_pos, "i32", "draft_pos")
        a.lag = _ptr(lag, "i32", "lag")
    a.temperature = float(temperature)
    if temperature != 0.0:
        a.uniforms = _ptr(uniforms, "u64", "uniforms")
        a.sample_workspace = _ptr(sample_workspace, "u8", "sample_workspace")
        a.sample_workspace_bytes = sample_workspace.numel()
        a.draft_logits = _ptr(draft_logits, "bf16", "draft_logits", True)
        a.accept_uniforms = _ptr(accept_uniforms, "u64", "accept_uniforms",
                                 draft_logits is None)
    return a


def switchsd_step(args, workspace, stream=None):
    _check("switchsd_step", lib.switchsd_step(ctypes.byref(args), _ptr(workspace, "u8",
                                              "workspace"), workspace.numel(),
                                              _stream(stream)))


def switchsd_step_noalloc(args, stream=None):
    """switchsd_step with the library's own fixed device scratch (no workspace
    argument; args.sample_workspace is ignored)."""
    _check("switchsd_step_noalloc", lib.switchsd_step_noalloc(ctypes.byref(args),
                                                              _stream(stream)))
