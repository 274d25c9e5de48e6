"""Build step for the CPU oracle: ``python -m oracle.build``.

Plain C, -O2, OpenMP, no fast-math (the oracle's floating point must follow
IEEE double semantics).
"""
from __future__ import annotations

import os
import subprocess
import sys

_HERE = os.path.dirname(os.path.abspath(__file__))


def build(verbose: bool = False, sanitize: bool = False, out: str | None = None) -> str:
    """Builds libsg_oracle.so; with `sanitize`, an AddressSanitizer and
    UndefinedBehaviorSanitizer build (load it with gcc's libasan preloaded)."""
    src = os.path.join(_HERE, "sg_oracle.c")
    out = out or os.path.join(_HERE, "libsg_oracle.so")
    tmp = out + ".tmp%d" % os.getpid()
    opt = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined"] if sanitize else ["-O2"]
    cmd = ["gcc", "-std=c11", *opt, "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-fno-fast-math", src, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
