"""CPU oracle of SwitchSD's per-step speculation-control path.

TEST INFRASTRUCTURE ONLY.  This package is the checker of the HIP library:
only the test-suite, the smoke check and the benchmark's CPU-baseline leg
import it.  The product path never does, and it shares no code with it.

The arithmetic lives in ``switchsd_oracle.c`` (plain scalar C); this module
only marshals numpy arrays through ctypes.  Each function cites the passage
of the paper it follows (see the C source for the readings R1-R8, R13-R15).
"""
import ctypes
import os

import numpy as np

from . import build_oracle

_lib = None

MAX_NGRAM = 8


class OracleCfg(ctypes.Structure):
    _fields_ = [("n_ngram", ctypes.c_int32),
                ("ngram_lens", ctypes.c_int32 * MAX_NGRAM),
                ("kappa", ctypes.c_int32),
                ("k", ctypes.c_int32),
                ("theta", ctypes.c_float),
                ("n_cand", ctypes.c_int32)]


def make_cfg(ngram_lens, kappa, k, theta, n_cand=1):
    c = OracleCfg()
    c.n_ngram = len(ngram_lens)
    for i, n in enumerate(ngram_lens):
        c.ngram_lens[i] = int(n)
    c.kappa = int(kappa)
    c.k = int(k)
    c.theta = float(theta)
    c.n_cand = int(n_cand)
    return c


def n_cand_of(cfg):
    """W: candidates per sequence (0 or 1 both mean one)."""
    return max(1, int(cfg.n_cand))


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(build_oracle.LIB):
            build_oracle.build()
        _lib = ctypes.CDLL(build_oracle.LIB)
        P = ctypes.c_void_p
        i32 = ctypes.c_int32
        _lib.oracle_match.argtypes = [P, i32, P, P, P, P, P]
        _lib.oracle_probe.argtypes = [P, P, i32, ctypes.c_float]
        _lib.oracle_probe.restype = ctypes.c_float
        _lib.oracle_match.restype = ctypes.c_int
        _lib.oracle_select.argtypes = [i32, P, P, ctypes.c_float, P, P, i32, i32, P, P, P, P]
        _lib.oracle_select.restype = i32
        _lib.oracle_argmax_row.argtypes = [P, i32]
        _lib.oracle_argmax_row.restype = i32
        _lib.oracle_accept.argtypes = [P, P, i32, P, i32, P, P, P, P]
        _lib.oracle_tree_mask.argtypes = [P, i32, i32, i32, P]
        _lib.oracle_step.argtypes = [i32, i32, i32, i32, i32] + [P] * 4 + [ctypes.c_float] + \
            [P] * 5 + [P] * 14 + [ctypes.c_float, P, P, P, i32]
        _lib.oracle_commit.argtypes = [P, P, i32, P, i32, i32, P, P]
        _lib.oracle_copy_labels.argtypes = [P, i32, i32, i32, P]
        _lib.oracle_sample_scale.argtypes = [ctypes.c_float]
        _lib.oracle_sample_scale.restype = ctypes.c_float
        _lib.oracle_sample_weight.argtypes = [ctypes.c_float, ctypes.c_float, ctypes.c_float]
        _lib.oracle_sample_weight.restype = ctypes.c_uint64
        _lib.oracle_row_weights.argtypes = [P, i32, ctypes.c_float, P]
        _lib.oracle_row_weights.restype = ctypes.c_uint64
        _lib.oracle_sample_row.argtypes = [P, i32, ctypes.c_float, ctypes.c_uint64]
        _lib.oracle_sample_row.restype = i32
        _lib.oracle_step.restype = i32
        _lib.oracle_spec_accept.argtypes = [P, P, i32, ctypes.c_float, i32, ctypes.c_uint64]
        _lib.oracle_spec_accept.restype = i32
        _lib.oracle_residual_row.argtypes = [P, P, i32, ctypes.c_float, ctypes.c_uint64]
        _lib.oracle_residual_row.restype = i32
    return _lib


def _p(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def match(x, L, cfg):
    """Step 1 (Sec. 3.3): longest-first suffix n-gram match, W most recent ends.

    Returns (match_n, match_end[W], copy_len[W], copy_tokens[W, k]); with
    W = 1 the last three are scalars and a [k] row, as before.
    """
    lib = _load()
    W = n_cand_of(cfg)
    x = _c(x, np.int32)
    if x.size == 0:
        x = np.zeros(1, np.int32)
    mn = np.zeros(1, np.int32)
    me = np.zeros(W, np.int32)
    cl = np.zeros(W, np.int32)
    ct = np.full(W * max(cfg.k, 1), -1, np.int32)
    lib.oracle_match(_p(x), int(L), ctypes.byref(cfg), _p(mn), _p(me), _p(cl), _p(ct))
    ct = ct[:W * cfg.k].reshape(W, cfg.k).copy()
    if cfg.n_cand <= 1:
        return int(mn[0]), int(me[0]), int(cl[0]), ct[0]
    return int(mn[0]), me, cl, ct


def probe(h_bf16, w, bias):
    """Step 2 (Sec. 3.2, Eq. 3): z = w . h + bias, rounded once to float."""
    lib = _load()
    h = _c(h_bf16, np.uint16)
    w = _c(w, np.float32)
    return np.float32(lib.oracle_probe(_p(h), _p(w), int(h.size), float(bias)))


def select(match_n, copy_len, copy_tokens, z, ntok, npar, nn, R, cfg):
    """Step 3 (Sec. 3.3, Eq. 4 + kappa gate): chosen draft in node layout."""
    lib = _load()
    W = n_cand_of(cfg)
    cl = _c(np.reshape(copy_len, (-1,)), np.int32)
    assert cl.size == W
    ct = _c(copy_tokens, np.int32).reshape(-1) if cfg.k > 0 else np.zeros(1, np.int32)
    ntok = _c(ntok, np.int32)
    npar_a = _c(npar, np.int32) if npar is not None else None
    dtok = np.zeros(R, np.int32)
    dpar = np.zeros(R, np.int32)
    dn = np.zeros(1, np.int32)
    uc = lib.oracle_select(int(match_n), _p(cl), _p(ct), float(z), _p(ntok), _p(npar_a),
                           int(nn), int(R), ctypes.byref(cfg), _p(dtok), _p(dpar), _p(dn))
    return int(uc), dtok, dpar, int(dn[0])


def argmax_row(row_bf16):
    """Step 4a (Sec. 2; App. A, T = 0): lowest index of the largest value."""
    lib = _load()
    r = _c(row_bf16, np.uint16)
    return int(lib.oracle_argmax_row(_p(r), int(r.size)))


def sample_scale(temperature):
    """c = log2(e) / T rounded to float (App. A, sampling temperature)."""
    return np.float32(_load().oracle_sample_scale(float(temperature)))


def sample_weight(l, m, c):
    """Integer weight floor(2^40 * 2^((l - m) c)) of one logit (see the C source)."""
    return int(_load().oracle_sample_weight(float(l), float(m), float(c)))


def row_weights(row_bf16, temperature):
    """The integer weights of a row (uint64 [V]) and their sum Z (App. A)."""
    lib = _load()
    r = _c(row_bf16, np.uint16)
    w = np.zeros(max(r.size, 1), np.uint64)
    Z = lib.oracle_row_weights(_p(r), int(r.size), float(sample_scale(temperature)), _p(w))
    return w[:r.size], int(Z)


def sample_row(row_bf16, temperature, u):
    """Token drawn from softmax(l / T) by inverse CDF with the 64-bit uniform u."""
    lib = _load()
    r = _c(row_bf16, np.uint16)
    return int(lib.oracle_sample_row(_p(r), int(r.size), float(sample_scale(temperature)),
                                     int(u)))


def spec_accept(p_row, q_row, temperature, x, u):
    """Speculative-sampling test (Sec. 2; App. A): is the drafted token x
    accepted at a row with target logits p_row and draft logits q_row, with
    the 64-bit uniform u?  (u Q_x Zp < 2^64 P_x Zq.)"""
    lib = _load()
    pr, qr = _c(p_row, np.uint16), _c(q_row, np.uint16)
    assert pr.size == qr.size
    return bool(lib.oracle_spec_accept(_p(pr), _p(qr), int(pr.size),
                                       float(sample_scale(temperature)), int(x), int(u)))


def residual_row(p_row, q_row, temperature, u):
    """Token drawn from the normalized residual max(0, p - q) with the 64-bit
    uniform u (Sec. 2; App. A)."""
    lib = _load()
    pr, qr = _c(p_row, np.uint16), _c(q_row, np.uint16)
    assert pr.size == qr.size
    return int(lib.oracle_residual_row(_p(pr), _p(qr), int(pr.size),
                                       float(sample_scale(temperature)), int(u)))


def accept(dtok, dpar, dn, amax, R):
    """Step 4b (Sec. 3.3): deepest accepted node, its path and the bonus."""
    lib = _load()
    dtok = _c(dtok, np.int32)
    dpar = _c(dpar, np.int32)
    amax = _c(amax, np.int32)
    al, an, bo = (np.zeros(1, np.int32) for _ in range(3))
    out = np.zeros(R, np.int32)
    lib.oracle_accept(_p(dtok), _p(dpar), int(dn), _p(amax), int(R), _p(al), _p(an), _p(bo),
                      _p(out))
    return int(al[0]), int(an[0]), int(bo[0]), out


def tree_mask(dpar, dn, R, words=None):
    """Sec. 3.3 (block-triangular attention): ancestor-or-self bit rows.

    Returns uint32 [R, words]; bit j of row i is set iff node j is on node i's
    path to the anchor (itself included).
    """
    lib = _load()
    if words is None:
        words = (R + 31) // 32
    dpar = _c(dpar, np.int32)
    m = np.zeros((R, words), np.uint32)
    lib.oracle_tree_mask(_p(dpar), int(dn), int(R), int(words), _p(m))
    return m


def commit(tokens, lengths, draft_pos, res):
    """Sec. 3.3 (KV Cache Synchronization): append every sequence's accepted
    tokens and bonus (res from step()) to tokens/lengths in place and update
    draft_pos; returns lag [B]."""
    lib = _load()
    B, Lmax = tokens.shape
    assert tokens.dtype == np.int32 and tokens.flags.c_contiguous
    lag = np.zeros(B, np.int32)
    for b in range(B):
        ln = np.array([lengths[b]], np.int32)
        dp = np.array([draft_pos[b]], np.int32)
        lg = np.zeros(1, np.int32)
        out = _c(res["out_tokens"][b], np.int32)
        row = tokens[b]
        lib.oracle_commit(_p(row), _p(ln), int(Lmax), _p(out), int(res["accept_len"][b]),
                          int(res["use_copy"][b]), _p(dp), _p(lg))
        lengths[b], draft_pos[b], lag[b] = ln[0], dp[0], lg[0]
    return lag


def copy_labels(tokens, lengths, n):
    """Sec. 3.2: copy-mode label of every position ([B, Lmax] uint8)."""
    lib = _load()
    tokens = _c(tokens, np.int32)
    B, Lmax = tokens.shape
    out = np.zeros((B, Lmax), np.uint8)
    for b in range(B):
        L = max(0, min(int(lengths[b]), Lmax))
        row = out[b]
        lib.oracle_copy_labels(_p(tokens[b]), L, Lmax, int(n), _p(row))
    return out


STEP_OUTPUTS = ("match_n", "match_end", "copy_len", "copy_tokens", "z", "use_copy",
                "dtok", "dpar", "dn", "amax", "accept_len", "accept_node", "bonus",
                "out_tokens")


def step(tokens, lengths, hidden, w, bias, ntok, npar, nn, logits, cfg, threads=1,
         temperature=0.0, uniforms=None, draft_logits=None, accept_uniforms=None):
    """The whole step for B sequences (steps 1-4 in the paper's order).

    tokens [B,Lmax] int32, lengths [B] int32, hidden [B,d] bf16 bits (uint16),
    w [d] float32, ntok/npar [B,R] int32 (npar None = chains), nn [B] int32,
    logits [B,R,V] bf16 bits (uint16).  temperature > 0 draws each row's
    token with uniforms [B,R] uint64 (App. A); amax then holds the drawn
    tokens.  draft_logits [B,R,V] bf16 bits (chains, T > 0) with
    accept_uniforms [B,R] uint64: sequences verifying their neural draft use
    speculative sampling with that draft distribution (see the C header).
    Returns a dict of numpy outputs.
    """
    lib = _load()
    tokens = _c(tokens, np.int32)
    B, Lmax = tokens.shape
    lengths = _c(lengths, np.int32)
    hidden = _c(hidden, np.uint16).reshape(B, -1)
    d = hidden.shape[1]
    w = _c(w, np.float32)
    ntok = _c(ntok, np.int32)
    R = ntok.shape[1]
    npar_a = _c(npar, np.int32) if npar is not None else None
    nn = _c(nn, np.int32)
    logits = _c(logits, np.uint16)
    V = logits.shape[-1]
    assert logits.size == B * R * V
    K = cfg.k
    W = n_cand_of(cfg)
    o = {
        "match_n": np.zeros(B, np.int32), "match_end": np.zeros((B, W), np.int32),
        "copy_len": np.zeros((B, W), np.int32),
        "copy_tokens": np.zeros((B, W, max(K, 1)), np.int32),
        "z": np.zeros(B, np.float32), "use_copy": np.zeros(B, np.int32),
        "dtok": np.zeros((B, R), np.int32), "dpar": np.zeros((B, R), np.int32),
        "dn": np.zeros(B, np.int32), "amax": np.zeros((B, R), np.int32),
        "accept_len": np.zeros(B, np.int32), "accept_node": np.zeros(B, np.int32),
        "bonus": np.zeros(B, np.int32), "out_tokens": np.zeros((B, R), np.int32),
    }
    un = _c(uniforms, np.uint64) if uniforms is not None else None
    if temperature > 0:
        assert un is not None and un.size == B * R
    ql = _c(draft_logits, np.uint16) if draft_logits is not None else None
    ua = _c(accept_uniforms, np.uint64) if accept_uniforms is not None else None
    if ql is not None:
        assert ql.size == B * R * V and ua is not None and ua.size == B * R
    rc = lib.oracle_step(B, Lmax, d, R, V, _p(tokens), _p(lengths), _p(hidden), _p(w),
                         float(bias), _p(ntok), _p(npar_a), _p(nn), _p(logits),
                         ctypes.byref(cfg), *[_p(o[k]) for k in STEP_OUTPUTS],
                         float(temperature), _p(un), _p(ql), _p(ua), int(threads))
    if rc != 0:
        raise ValueError("oracle_step rejected its arguments")
    o["copy_tokens"] = o["copy_tokens"][:, :, :K]
    if cfg.n_cand <= 1:
        o["match_end"] = o["match_end"][:, 0].copy()
        o["copy_len"] = o["copy_len"][:, 0].copy()
        o["copy_tokens"] = o["copy_tokens"][:, 0].copy()
    return o


def front(tokens, lengths, hidden, w, bias, ntok, npar, nn, cfg):
    """Steps 1-3 for every sequence (match, probe, switch), no logits needed."""
    tokens = _c(tokens, np.int32)
    B, Lmax = tokens.shape
    R = ntok.shape[1]
    W = n_cand_of(cfg)
    wsh = (B,) if cfg.n_cand <= 1 else (B, W)
    o = {k: np.zeros(B, np.int32) for k in ("match_n", "use_copy", "dn")}
    o["match_end"] = np.zeros(wsh, np.int32)
    o["copy_len"] = np.zeros(wsh, np.int32)
    o["z"] = np.zeros(B, np.float32)
    o["copy_tokens"] = np.zeros(wsh + (cfg.k,), np.int32)
    o["dtok"] = np.zeros((B, R), np.int32)
    o["dpar"] = np.zeros((B, R), np.int32)
    for b in range(B):
        L = max(0, min(int(lengths[b]), Lmax))
        mn, me, cl, ct = match(tokens[b], L, cfg)
        z = probe(hidden[b], w, bias)
        uc, dtok, dpar, dn = select(mn, cl, ct, z, ntok[b], None if npar is None else npar[b],
                                    nn[b], R, cfg)
        o["match_n"][b], o["match_end"][b], o["copy_len"][b] = mn, me, cl
        o["copy_tokens"][b] = ct
        o["z"][b], o["use_copy"][b], o["dn"][b] = z, uc, dn
        o["dtok"][b], o["dpar"][b] = dtok, dpar
    return o
