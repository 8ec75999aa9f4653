"""Host logic of bench.py (no GPU): the one-GPU guard, the launch AUTO picks,
and the algorithmic byte count behind the roofline figure."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2609_20186_amd import workloads as W  # noqa: E402


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr or "single MI355X" in r.stderr


def test_auto_mode_matches_the_library_rule():
    # one launch when every row may be needed (1 + W k >= R) and R <= 64
    fused = {n for n, wl in W.WORKLOADS.items() if bench.resolve_mode(wl, 0) == 1}
    assert fused == {"C1", "C2", "C3", "C4"}
    assert bench.resolve_mode(W.WORKLOADS["C5"], 0) == 2
    assert bench.resolve_mode(W.WORKLOADS["C2W10"], 0) == 2
    assert bench.resolve_mode(W.WORKLOADS["C5"], 1) == 1   # an explicit mode is kept


def test_c2_algorithmic_bytes():
    wl = W.WORKLOADS["C2"]
    total, logits = bench.algorithmic_bytes(wl, np.full(wl.B, wl.R))
    # the scope table's inputs: tokens, hidden states, probe weight, logits
    assert logits == 32 * 8 * 128256 * 2 == 65_667_072
    core = 32 * 4096 * 4 + 32 * 4096 * 2 + 4096 * 4 + logits
    assert core == 66_469_888
    # plus lengths, the neural draft and its sizes, and the int32 outputs
    assert core < total < core + 16_384
    assert logits / total > 0.987
    # a split step counts only the drafted rows
    _, part = bench.algorithmic_bytes(wl, np.full(wl.B, 3))
    assert part == 32 * 3 * 128256 * 2


def test_every_name_bench_calls_is_defined():
    """Every bare name bench.py calls is a builtin, an import or a definition
    of the script (the decode-loop option once called a function that a
    rewrite had dropped)."""
    import ast
    import builtins
    src = open(os.path.join(ROOT, "bench.py")).read()
    tree = ast.parse(src)
    known = set(dir(builtins))
    for node in ast.walk(tree):
        if isinstance(node, (ast.FunctionDef, ast.ClassDef)):
            known.add(node.name)
            known.update(a.arg for a in node.args.args + node.args.kwonlyargs) \
                if isinstance(node, ast.FunctionDef) else None
        elif isinstance(node, (ast.Import, ast.ImportFrom)):
            known.update((a.asname or a.name).split(".")[0] for a in node.names)
        elif isinstance(node, ast.Name) and isinstance(node.ctx, ast.Store):
            known.add(node.id)
        elif isinstance(node, ast.arg):
            known.add(node.arg)
    called = {n.func.id for n in ast.walk(tree)
              if isinstance(n, ast.Call) and isinstance(n.func, ast.Name)}
    assert not called - known, sorted(called - known)
