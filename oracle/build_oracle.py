"""Compile the oracle's C GEMM (``gemm_fp64.c``) into ``liboracle_gemm.so``.

Plain ``gcc -O2 -fopenmp``; no vector intrinsics, no blocking.
"""

import os
import subprocess

_HERE = os.path.dirname(os.path.abspath(__file__))


def build(verbose=False):
    src = os.path.join(_HERE, "gemm_fp64.c")
    out = os.path.join(_HERE, "liboracle_gemm.so")
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-Wall", "-Werror",
           src, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
