"""Compile the CPU oracle (oracle/wfref.c) into oracle/libwfref.so with gcc.

Test infrastructure only: the oracle is built so the tests, the smoke check
and the benchmark's CPU-baseline leg can run it.  No product code links it.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "wfref.c")
LIB = os.path.join(HERE, "libwfref.so")


SAN_FLAGS = ["-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=undefined"]


def build(verbose: bool = False, out: str = None, sanitize: bool = False) -> str:
    """Compile the oracle; returns the path of the shared library.  With
    sanitize=True the library is built with AddressSanitizer and
    UndefinedBehaviorSanitizer (run it with gcc's libasan preloaded)."""
    lib = out or LIB
    tmp = lib + ".tmp"
    cmd = ["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared",
           "-Wall", "-Wextra"] + (SAN_FLAGS if sanitize else []) + \
        ["-o", tmp, SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose=True))
