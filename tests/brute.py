"""A second, independent formulation of the step for tiny inputs.

Used only to pin the C oracle.  Each piece is phrased differently from the
oracle's scalar loops, on purpose:

* match  -- a byte-string search (``bytes.rfind``) of the suffix's
            little-endian encoding, re-checked for 4-byte alignment;
* probe  -- ``math.fsum`` of the exact products (correctly rounded double),
            then one rounding to float32;
* argmax -- ``numpy`` max over the non-NaN entries, then the first index
            equal to it;
* accept -- for every node, walk its path up to the root and test each
            edge; keep the deepest node whose whole path holds.

Paper: Sec. 3.3 (kappa-gram gate, recency ranking, Eq. 4, longest validated
continuation), Sec. 3.2 Eq. 3 (linear probe), Sec. 2 and App. A (greedy
verification at T = 0).
"""
import math

import numpy as np


def bf16_to_f32(h):
    return (np.asarray(h, np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def match_all(x, L, lens, k, W):
    """The W most recent occurrences of the longest matching suffix length.

    Returns (n, ends[W], lens[W], tokens[W][k]) padded with -1 / 0 / -1.
    """
    x = np.asarray(x[:L], dtype="<i4")
    for n in lens:
        if L < n + 1:
            continue
        pat = x[L - n:].tobytes()
        hay = x[:L - 1].tobytes()          # occurrences must end at e <= L-2
        pos = len(hay)
        starts = []
        while len(starts) < W:
            i = hay.rfind(pat, 0, pos)
            if i < 0:
                break
            if i % 4 == 0:
                starts.append(i // 4)
            pos = i + len(pat) - 1      # retry strictly before this hit's end
        if starts:
            ends, cls, cts = [], [], []
            for s0 in starts:
                e = s0 + n - 1
                c = e + 1
                cl = min(k, L - c)
                ends.append(e)
                cls.append(cl)
                cts.append([int(t) for t in x[c:c + cl]] + [-1] * (k - cl))
            pad = W - len(starts)
            return (n, ends + [-1] * pad, cls + [0] * pad, cts + [[-1] * k] * pad)
    return 0, [-1] * W, [0] * W, [[-1] * k] * W


def match(x, L, lens, k):
    n, ends, cls, cts = match_all(x, L, lens, k, 1)
    return n, ends[0], cls[0], cts[0]


def probe(h_bf16, w, bias):
    hf = bf16_to_f32(h_bf16).astype(np.float64)
    wf = np.asarray(w, np.float32).astype(np.float64)
    terms = [float(a) * float(b) for a, b in zip(hf, wf)]   # exact in double
    return np.float32(math.fsum(terms + [float(np.float32(bias))]))


def argmax_row(row_bf16):
    f = bf16_to_f32(row_bf16)
    ok = np.flatnonzero(~np.isnan(f))
    if ok.size == 0:
        return 0
    m = f[ok].max()
    return int(np.flatnonzero(f == m)[0])


def select(match_n, copy_len, copy_tokens, z, ntok, npar, nn, R, kappa, theta):
    dtok = [-1] * R
    dpar = [-1] * R
    if match_n >= kappa and np.float32(z) >= np.float32(theta):
        if np.ndim(copy_len) == 0:                  # one candidate
            copy_len, copy_tokens = [copy_len], [copy_tokens]
        nodes = [(0, -1)]                           # (token, parent); anchor first
        for cl, ct in zip(copy_len, copy_tokens):
            for i in range(int(cl)):
                nodes.append((int(ct[i]), 0 if i == 0 else len(nodes) - 1))
        for i, (t, par) in enumerate(nodes[1:], start=1):
            dtok[i], dpar[i] = t, par
        return 1, dtok, dpar, len(nodes)
    nn = max(1, min(int(nn), R))
    for i in range(1, nn):
        dtok[i] = int(ntok[i])
        dpar[i] = int(npar[i]) if npar is not None else i - 1
    return 0, dtok, dpar, nn


def accept(dtok, dpar, dn, amax, R):
    best, best_depth, best_path = 0, 0, []
    for i in range(1, dn):
        path = [i]
        ok = True
        while path[-1] != 0:
            c = path[-1]
            p = int(dpar[c])
            if not (0 <= p < c) or int(dtok[c]) != int(amax[p]):
                ok = False
                break
            path.append(p)
        if ok and len(path) - 1 > best_depth:
            best, best_depth, best_path = i, len(path) - 1, path
    toks = [int(dtok[n]) for n in reversed(best_path[:-1])] if best_path else []
    bonus = int(amax[best])
    out = toks + [bonus] + [-1] * (R - len(toks) - 1)
    return best_depth, best, bonus, out


def tree_mask(dpar, dn, R):
    """Ancestor-or-self sets as Python sets (a node with a bad parent stops)."""
    rows = []
    for i in range(R):
        s = set()
        if i < dn:
            c = i
            s.add(c)
            while c != 0 and 0 <= int(dpar[c]) < c:
                c = int(dpar[c])
                s.add(c)
        rows.append(s)
    return rows


def step(tokens, lengths, hidden, w, bias, ntok, npar, nn, logits, lens, kappa, k, theta,
         n_cand=1):
    W = max(1, n_cand)
    B, Lmax = tokens.shape
    R = ntok.shape[1]
    res = {key: [] for key in ("match_n", "match_end", "copy_len", "copy_tokens", "z",
                               "use_copy", "dtok", "dpar", "dn", "amax", "accept_len",
                               "accept_node", "bonus", "out_tokens")}
    for b in range(B):
        L = max(0, min(int(lengths[b]), Lmax))
        if n_cand <= 1:
            mn, me, cl, ct = match(tokens[b], L, lens, k)
        else:
            mn, me, cl, ct = match_all(tokens[b], L, lens, k, W)
        z = probe(hidden[b], w, bias)
        uc, dtok, dpar, dn = select(mn, cl, ct, z, ntok[b], None if npar is None else npar[b],
                                    nn[b], R, kappa, theta)
        amax = [argmax_row(logits[b, r]) if r < dn else -1 for r in range(R)]
        al, an, bo, out = accept(dtok, dpar, dn, amax, R)
        for key, v in zip(res, (mn, me, cl, ct, z, uc, dtok, dpar, dn, amax, al, an, bo, out)):
            res[key].append(v)
    out = {}
    for key, v in res.items():
        out[key] = np.asarray(v, np.float32 if key == "z" else np.int32)
    out["copy_tokens"] = out["copy_tokens"].reshape((B, k) if n_cand <= 1 else (B, W, k))
    return out
