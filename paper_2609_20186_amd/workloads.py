"""Seeded synthetic inputs for SwitchSD's speculation-control step.

This module draws inputs and nothing else: it holds none of the method's
arithmetic (no n-gram search, no probe, no switch, no argmax, no accept).
Both the HIP path's tests/benchmark and the CPU oracle take their inputs
from here.  ``plant`` shapes the logits so that a given draft is accepted up
to a chosen node; the draft it plants for is an argument supplied by the
caller.

The paper's evaluation suites (HumanEval, Math500, CNN/DailyMail, MT-Bench)
and its models are not available, so five synthetic workloads stand in for
them, with the shapes of the models the paper evaluates (Sec. 4) and the
copy regimes it describes (Sec. 3.1: accidental repetitions; Fig. 2):

  C1 tiny chain step          B=1   L=512    V=32000   d=1024 k=5
  C2 Llama-3-8B copy-heavy    B=32  L=4096   V=128256  d=4096 k=7
  C3 Qwen-14B low-copy        B=64  L=8192   V=151936  d=5120 k=7  bias=-2
  C4 long-context edit        B=8   L=32768  V=128256  d=8192 k=10
  C5 tree verification        B=256 L=2048   V=128256  d=4096 k=7  60-node tree

Every array of sequence b is drawn from its own numpy PCG64 stream
``SeedSequence([20186, cfg_id, stream, b])``, so any subset of a batch can be
regenerated on its own.
"""
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass
from functools import lru_cache
import math
import os

import numpy as np

BF16_PLUS8 = 0x4100   # bf16 bits of +8.0 (above the +-7.5 clamp of the noise)
BF16_MINUS8 = 0xC100  # bf16 bits of -8.0

S_TOKENS, S_HIDDEN, S_DRAFT, S_LOGITS, S_PLANT, S_W, S_TREE = range(7)


@dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int
    B: int
    L: int
    V: int
    d: int
    k: int
    R: int
    ngram_lens: tuple = (3, 2, 1)
    kappa: int = 1
    bias: float = 0.0
    theta: float = 0.0           # logit(tau); tau = 0.5
    context: str = "spans"       # "c1" | "spans" | "iid"
    zipf_s: float = 1.1
    span_frac: float = 0.0
    span_len: tuple = (0, 0)
    subst: float = 0.0
    draft: str = "zipf_chain"    # "uniform_chain" | "zipf_chain" | "tree"
    tree_nodes: int = 0
    tree_depth: int = 0
    plant: str = "copy_full_neural_geom"   # | "uniform" | "geom"
    geom_p: float = 0.6
    n_cand: int = 1              # copy candidates W
    neural_k: int = 0            # neural chain length (0: k)
    cand_p: float = 0.5          # accepted copy candidate c: P(c >= j) = cand_p^j

    @property
    def chain(self):
        return self.draft != "tree"

    def logits_bytes(self):
        return self.B * self.R * self.V * 2


WORKLOADS = {
    "C1": Workload("C1", 1, B=1, L=512, V=32000, d=1024, k=5, R=6, context="c1",
                   draft="uniform_chain", plant="uniform"),
    "C2": Workload("C2", 2, B=32, L=4096, V=128256, d=4096, k=7, R=8, context="spans",
                   zipf_s=1.1, span_frac=0.3, span_len=(32, 256), geom_p=0.6),
    "C3": Workload("C3", 3, B=64, L=8192, V=151936, d=5120, k=7, R=8, context="iid",
                   zipf_s=1.05, bias=-2.0, plant="geom", geom_p=0.5),
    "C4": Workload("C4", 4, B=8, L=32768, V=128256, d=8192, k=10, R=11, context="spans",
                   zipf_s=1.1, span_frac=0.6, span_len=(128, 2048), subst=0.01, geom_p=0.6),
    "C5": Workload("C5", 5, B=256, L=2048, V=128256, d=4096, k=7, R=60, context="spans",
                   zipf_s=1.1, span_frac=0.2, span_len=(16, 128), draft="tree",
                   tree_nodes=60, tree_depth=7, geom_p=0.6),
    # the paper's copy setting (W = 10 candidates of D = 20 tokens, Sec. 3.3 and
    # App. D) on the C2 context and vocabulary, with a 7-token neural chain
    "C2W10": Workload("C2W10", 6, B=32, L=4096, V=128256, d=4096, k=20, R=201,
                      context="spans", zipf_s=1.1, span_frac=0.3, span_len=(32, 256),
                      geom_p=0.6, n_cand=10, neural_k=7),
}


def rng_for(wl, stream, b=None):
    key = [20186, wl.cfg_id, stream] + ([] if b is None else [int(b)])
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(key)))


def f32_to_bf16_bits(f):
    """Round float32 values to bf16 (round to nearest, ties to even); finite input."""
    u = np.ascontiguousarray(f, dtype=np.float32).view(np.uint32)
    return ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(h):
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@lru_cache(maxsize=8)
def _zipf_cdf(s, V):
    p = np.arange(1, V + 1, dtype=np.float64) ** (-s)
    c = np.cumsum(p)
    return c / c[-1]


def zipf_tokens(rng, n, s, V):
    """Truncated Zipf over ranks 1..V (P(r) ~ r^-s); token id = rank - 1."""
    u = rng.random(n)
    return np.minimum(np.searchsorted(_zipf_cdf(s, V), u, side="right"), V - 1).astype(np.int32)


def span_start_prob(wl):
    mean_len = 0.5 * (wl.span_len[0] + wl.span_len[1])
    f = wl.span_frac
    return f / (mean_len * (1.0 - f) + f)


def make_context(wl, b):
    """One context of length L (int32 token ids in [0, V))."""
    rng = rng_for(wl, S_TOKENS, b)
    L, V = wl.L, wl.V
    if wl.context == "c1":
        # uniform tokens; a 64-token window [s, s+64) whose first 64-r tokens are
        # repeated at the very end, so the context stops in the middle of a copy
        x = rng.integers(0, V, L, dtype=np.int64).astype(np.int32)
        r = int(rng.integers(5, 33))
        s = int(rng.integers(0, L - 128 + r + 1))
        m = 64 - r
        x[L - m:] = x[s:s + m]
        return x
    x = zipf_tokens(rng, L, wl.zipf_s, V)
    if wl.context == "iid":
        return x
    q = span_start_prob(wl)
    lo, hi = wl.span_len
    p = 0
    while True:
        p += int(rng.geometric(q)) - 1
        if p >= L:
            break
        ln = min(int(rng.integers(lo, hi + 1)), L - p, p)
        if ln <= 0:
            p += 1
            continue
        src = int(rng.integers(0, p - ln + 1))
        x[p:p + ln] = x[src:src + ln]
        if wl.subst > 0:
            hit = rng.random(ln) < wl.subst
            nsub = int(hit.sum())
            if nsub:
                x[p:p + ln][hit] = rng.integers(0, V, nsub).astype(np.int32)
        p += ln
    return x


@lru_cache(maxsize=4)
def tree_parents(wl):
    """Seeded parent array of the neural token tree (node 0 = root, parent < i,
    depth <= tree_depth), shared by every sequence of the workload."""
    rng = rng_for(wl, S_TREE)
    par = np.full(wl.tree_nodes, -1, np.int32)
    depth = np.zeros(wl.tree_nodes, np.int32)
    for i in range(1, wl.tree_nodes):
        cand = np.flatnonzero(depth[:i] <= wl.tree_depth - 1)
        p = int(cand[rng.integers(0, cand.size)])
        par[i] = p
        depth[i] = depth[p] + 1
    return par


def make_neural_draft(wl, b):
    """(ntok[R], npar[R] or None, nn) -- the neural draft as the drafter hands it
    over (the paper delegates it to SPS or EAGLE3, Sec. 3.3)."""
    rng = rng_for(wl, S_DRAFT, b)
    R = wl.R
    ntok = np.full(R, -1, np.int32)
    kn = wl.neural_k or wl.k
    if wl.draft == "uniform_chain":
        ntok[1:kn + 1] = rng.integers(0, wl.V, kn)
        return ntok, None, kn + 1
    if wl.draft == "zipf_chain":
        ntok[1:kn + 1] = zipf_tokens(rng, kn, wl.zipf_s, wl.V)
        return ntok, None, kn + 1
    par = tree_parents(wl).copy()
    n = wl.tree_nodes
    for i in range(1, n):
        sib = set(int(ntok[j]) for j in range(1, i) if par[j] == par[i])
        while True:
            t = int(zipf_tokens(rng, 1, wl.zipf_s, wl.V)[0])
            if t not in sib:
                break
        ntok[i] = t
    npar = np.full(R, -1, np.int32)
    npar[:n] = par
    return ntok, npar, n


def make_logits_rows(wl, b):
    """[R, V] bf16 bits: N(0,1) clamped to [-7.5, 7.5], rounded to bf16."""
    rng = rng_for(wl, S_LOGITS, b)
    f = rng.standard_normal((wl.R, wl.V), dtype=np.float32)
    np.clip(f, -7.5, 7.5, out=f)
    return f32_to_bf16_bits(f)


def generate(wl, batch=None, logits=True):
    """Inputs of workload ``wl`` for the sequences in ``batch`` (default: all).

    Returns a dict with tokens [n,L] int32, lengths [n] int32, hidden [n,d]
    uint16 (bf16 bits), w [d] float32, ntok [n,R] int32, npar [n,R] int32 or
    None, nn [n] int32 and (if ``logits``) logits [n,R,V] uint16 (unplanted).
    """
    if isinstance(wl, str):
        wl = WORKLOADS[wl]
    idx = list(range(wl.B)) if batch is None else [int(b) for b in batch]
    n = len(idx)
    tokens = np.empty((n, wl.L), np.int32)
    hidden = np.empty((n, wl.d), np.uint16)
    ntok = np.empty((n, wl.R), np.int32)
    npar = None if wl.chain else np.empty((n, wl.R), np.int32)
    nn = np.empty(n, np.int32)
    lg = np.empty((n, wl.R, wl.V), np.uint16) if logits else None
    for j, b in enumerate(idx):
        tokens[j] = make_context(wl, b)
        hidden[j] = f32_to_bf16_bits(rng_for(wl, S_HIDDEN, b).standard_normal(wl.d, dtype=np.float32))
        t, p, c = make_neural_draft(wl, b)
        ntok[j] = t
        if npar is not None:
            npar[j] = p
        nn[j] = c
    if logits:
        def fill(j):
            lg[j] = make_logits_rows(wl, idx[j])
        workers = max(1, min(16, os.cpu_count() or 1, n))
        if workers > 1 and n * wl.R * wl.V > (1 << 24):
            with ThreadPoolExecutor(workers) as ex:
                list(ex.map(fill, range(n)))
        else:
            for j in range(n):
                fill(j)
    w = (rng_for(wl, S_W).standard_normal(wl.d) / math.sqrt(wl.d)).astype(np.float32)
    return {"tokens": tokens, "lengths": np.full(n, wl.L, np.int32), "hidden": hidden,
            "w": w, "bias": np.float32(wl.bias), "ntok": ntok, "npar": npar, "nn": nn,
            "logits": lg, "batch": np.asarray(idx, np.int64)}


def _children(dpar, dn, node):
    return [c for c in range(1, dn) if dpar[c] == node]


def draw_target(wl, b, dpar, dn, use_copy):
    """The node the planted logits should make the deepest accepted one."""
    rng = rng_for(wl, S_PLANT, b)
    last = dn - 1
    if wl.plant == "uniform":
        return int(rng.integers(0, min(wl.k, last) + 1))  # chains: node index = depth
    g = int(rng.geometric(1.0 - wl.geom_p)) - 1           # P(g >= j) = p^j
    if wl.plant == "geom":
        steps = g
    elif use_copy and wl.n_cand > 1:
        # one candidate accepted in full, the more recent ones more likely
        starts = _children(dpar, dn, 0)
        if not starts:
            return 0
        c = min(int(rng.geometric(1.0 - wl.cand_p)) - 1, len(starts) - 1)
        return starts[c + 1] - 1 if c + 1 < len(starts) else last
    elif use_copy:
        return last                                        # copy drafts: accepted in full
    else:
        steps = g
    if wl.chain or use_copy:
        return min(steps, last)
    node = 0
    for _ in range(min(steps, wl.tree_depth)):
        ch = _children(dpar, dn, node)
        if not ch:
            break
        node = int(ch[rng.integers(0, len(ch))])
    return node


def plant(logits_rows, dtok, dpar, dn, target):
    """Make ``target`` the deepest accepted node of the draft (dtok, dpar, dn).

    logits_rows is the [R, V] bf16 block of one sequence, modified in place:
    along the path root -> target, the parent's row gets +8.0 at the child's
    token (the strict row maximum); every child of the target gets -8.0 in the
    target's row.  Tokens outside [0, V) are left alone.
    """
    V = logits_rows.shape[1]
    node = int(target)
    while node > 0:
        p = int(dpar[node])
        t = int(dtok[node])
        if 0 <= t < V:
            logits_rows[p, t] = BF16_PLUS8
        node = p
    for c in _children(dpar, dn, int(target)):
        t = int(dtok[c])
        if 0 <= t < V:
            logits_rows[int(target), t] = BF16_MINUS8


def depth_of(dpar, node):
    d = 0
    while node > 0:
        node = int(dpar[node])
        d += 1
    return d


def plant_batch(wl, data, sel):
    """Plant every sequence of ``data`` for the drafts in ``sel`` (dicts with
    dtok [n,R], dpar [n,R], dn [n], use_copy [n]).  Returns the intended
    accepted node per sequence."""
    if isinstance(wl, str):
        wl = WORKLOADS[wl]
    n = data["tokens"].shape[0]
    tgt = np.zeros(n, np.int32)
    for j in range(n):
        b = int(data["batch"][j])
        dn = int(sel["dn"][j])
        t = draw_target(wl, b, sel["dpar"][j], dn, bool(sel["use_copy"][j]))
        plant(data["logits"][j], sel["dtok"][j], sel["dpar"][j], dn, t)
        tgt[j] = t
    return tgt
