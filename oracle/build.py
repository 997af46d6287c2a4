"""Compile the CPU oracle (oracle/wfref.c) into oracle/libwfref.so with gcc.

Test infrastructure only: the oracle is built so the tests, the smoke check
and the benchmark's CPU-baseline leg can run it.  No product code links it.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "wfref.c")
LIB = os.path.join(HERE, "libwfref.so")


def build(verbose: bool = False) -> str:
    """Compile the oracle; returns the path of the shared library."""
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared",
           "-Wall", "-Wextra", "-o", tmp, SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
