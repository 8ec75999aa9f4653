"""Build libswitchsd.so (HIP for gfx950) in-tree.

    python -m paper_2609_20186_amd.build

Compiles the kernels and the C entry points with hipcc for gfx950 and links
them into ``paper_2609_20186_amd/libswitchsd.so``.
"""
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libswitchsd.so")
TIMELINE_LIB = os.path.join(PKG, "libswitchsd_timeline.so")
CALIBRATE_LIB = os.path.join(PKG, "libswitchsd_calibrate.so")
BUILD = os.path.join(PKG, "_build")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
COMMON = ["-O3", "-std=c++17", "-fPIC", "-ffp-contract=off", "-Wall",
          "-I", INCLUDE, "-I", CSRC]
# packed fp32 VALU ops stay disabled in every device compile
DEVICE = ["--offload-arch=" + ARCH, "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
SOURCES = ["switchsd_kernels.hip", "switchsd_noalloc.hip", "switchsd_api.cpp"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError("build failed:\n" + " ".join(cmd) + "\n" + out)
    if verbose and out.strip():
        print(out)


def _link(objs, lib, verbose):
    tmp = lib + ".tmp"
    _run([HIPCC, "-shared", "--offload-arch=" + ARCH, "-fPIC", "-o", tmp] + objs, verbose)
    os.replace(tmp, lib)


def _compile(sources, subdir, defines, verbose):
    out = os.path.join(BUILD, subdir)
    os.makedirs(out, exist_ok=True)
    objs = []
    for src in sources:
        obj = os.path.join(out, src + ".o")
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        _run([HIPCC] + COMMON + defines + DEVICE + lang + ["-c", os.path.join(CSRC, src), "-o", obj],
             verbose)
        objs.append(obj)
    return objs


def build(verbose=False):
    """The step's library, then the two measurement builds: the same sources
    with per-work-group phase stamps (libswitchsd_timeline.so, used only by
    ``timeline.py``) and the streaming-read calibration kernel
    (libswitchsd_calibrate.so, used only by ``bench.py``)."""
    _link(_compile(SOURCES, "product", [], verbose), LIB, verbose)
    _link(_compile(SOURCES, "timeline", ["-DSWITCHSD_TIMELINE"], verbose), TIMELINE_LIB, verbose)
    _link(_compile(["read_calibration.hip"], "calibrate", [], verbose), CALIBRATE_LIB, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-q" not in sys.argv))
