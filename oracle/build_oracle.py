"""Compile the CPU oracle (plain C) into oracle/liboracle.so.

Test infrastructure: the oracle is the checker of the HIP path, never a part
of it.  Building it is not using it.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")


def build(verbose=False, sanitize=False):
    """sanitize: build with AddressSanitizer and UndefinedBehaviorSanitizer
    (host code; load it with the ASan runtime preloaded, e.g.
    ``LD_PRELOAD=$(gcc -print-file-name=libasan.so)``), for a checked run of
    the CPU tests."""
    src = os.path.join(HERE, "switchsd_oracle.c")
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-fno-omit-frame-pointer", "-g"] if sanitize else []
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared",
           "-pthread"] + san + ["-o", LIB + ".tmp", src, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    import sys
    print(build(verbose=True, sanitize="--sanitize" in sys.argv))
