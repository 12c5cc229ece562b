"""Build the CPU oracle (plain C, gcc) into oracle/libibp_oracle.so.

Test infrastructure only: the oracle is compiled so that the tests, the smoke check
and the benchmark's CPU-baseline leg can call it; the product library never links it.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "ibp_oracle.c")
LIB = os.path.join(HERE, "libibp_oracle.so")


def build(extra_flags=(), out=LIB, verbose=False):
    """Compile ibp_oracle.c with gcc. extra_flags lets a test build a variant."""
    cmd = ["gcc", "-O2", "-std=c99", "-Wall", "-Wextra", "-fPIC", "-shared",
           *extra_flags, SRC, "-o", out]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return out


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
