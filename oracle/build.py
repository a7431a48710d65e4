"""Build the CPU oracle library (test infrastructure only).

Compiles oracle/diffkv_oracle.c with gcc into oracle/liboracle_diffkv.so.
Strict IEEE fp32 (no contraction, no fast-math) so that the quantizer's
float arithmetic is exactly the arithmetic its comments describe.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "diffkv_oracle.c")
LIB = os.path.join(HERE, "liboracle_diffkv.so")


def build(verbose=False):
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-ffp-contract=off",
           "-fno-fast-math", "-fPIC", "-shared", SRC, "-o", LIB + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
