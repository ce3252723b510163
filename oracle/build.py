"""Build the fp64 reference-convolution library (test infrastructure only).

Compiles ``conv_oracle.c`` with gcc into ``liboracle_conv.so`` next to it.
Plain ``-O2`` with OpenMP; no fast-math, so every sum is evaluated in the
order the source writes it.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "conv_oracle.c")
OUT = os.path.join(HERE, "liboracle_conv.so")


def build(verbose=False):
    # a temporary name of this process's own, renamed into place: builds in
    # concurrent processes (parallel test workers) do not clobber each other
    tmp = f"{OUT}.{os.getpid()}.tmp"
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
           "-fno-fast-math", "-ffp-contract=off", SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose=True))
