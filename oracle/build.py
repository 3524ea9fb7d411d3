"""Compile the CPU oracle (pld_oracle.c) into oracle/libpld_oracle.so with gcc.

Test infrastructure: the oracle is never linked into the product library.
It is built without fast-math and with FMA contraction off, so every double
operation is one correctly rounded IEEE operation in source order.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "pld_oracle.c")
LIB = os.path.join(HERE, "libpld_oracle.so")


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-std=c11", "-O2", "-fPIC", "-shared", "-ffp-contract=off",
           "-fno-fast-math", "-Wall", "-Wextra", "-Werror", SRC, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
