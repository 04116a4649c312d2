"""Builds the CPU oracle library in place (plain C, no contraction, no fast-math)."""
from __future__ import annotations

import os
import subprocess

_HERE = os.path.dirname(os.path.abspath(__file__))


def compile_library(src: str, out: str, verbose: bool = False) -> str:
    """Compiles one oracle source file into a shared library at `out`."""
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared", src, "-lm", "-o",
           out + ".tmp"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    os.replace(out + ".tmp", out)
    return out


def build(verbose: bool = False) -> str:
    return compile_library(os.path.join(_HERE, "oracle.c"), os.path.join(_HERE, "liboracle.so"), verbose)


if __name__ == "__main__":
    build(verbose=True)
