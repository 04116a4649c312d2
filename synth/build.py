"""Builds the two twins of the synthetic-input generator in place."""
from __future__ import annotations

import os
import subprocess

_HERE = os.path.dirname(os.path.abspath(__file__))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# No packed-fp32 instructions in any GPU code of this repository.
NO_PACKED_FP32 = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def build_cpu(verbose: bool = False) -> str:
    out = os.path.join(_HERE, "libsynth_cpu.so")
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fPIC", "-shared",
           os.path.join(_HERE, "csrc", "synth_cpu.c"), "-o", out + ".tmp"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    os.replace(out + ".tmp", out)
    return out


def build_hip(verbose: bool = False) -> str:
    out = os.path.join(_HERE, "libsynth_hip.so")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-fPIC", "-shared", "-ffp-contract=off",
           *NO_PACKED_FP32, os.path.join(_HERE, "csrc", "synth_hip.hip"), "-o", out + ".tmp"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    os.replace(out + ".tmp", out)
    return out


def build(verbose: bool = False):
    build_cpu(verbose)
    build_hip(verbose)


if __name__ == "__main__":
    build(verbose=True)
