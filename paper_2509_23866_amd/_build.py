"""Build step for libdart.so (hipcc, gfx950). Always compiles when called."""

from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRCS = [os.path.join(HERE, "csrc", n) for n in ("dart.hip", "lmhead.hip", "check.hip")]
LIB = os.path.join(HERE, "libdart.so")
INCLUDE = os.path.join(ROOT, "include")

HIPCC_FLAGS = [
    "-O3", "--offload-arch=gfx950", "-std=c++17", "-fPIC", "-shared", "-Werror=shadow",
    # packed-FP32 VALU forms stay disabled: plain scalar fp32 code only
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def build(verbose: bool = False, extra_flags=(), out: str = LIB) -> str:
    cmd = ["hipcc", *HIPCC_FLAGS, *extra_flags, "-I", INCLUDE, *SRCS, "-o", out]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return out


if __name__ == "__main__":
    build(verbose=True)
