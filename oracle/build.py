"""Builds the oracle's shared library (host gcc, OpenMP).  Test infrastructure only."""
import os
import subprocess
import sys

ORACLE_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(ORACLE_DIR, "liboracle.so")


def build(verbose: bool = False, source: str = None, out: str = None) -> str:
    """Compiles oracle.c (or another source, e.g. a planted-mistake copy in a
    test) into a shared library; returns its path."""
    out = out or LIB_PATH
    tmp = out + ".tmp"
    cmd = ["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-std=c11", "-Wall", "-Wextra",
           "-o", tmp, source or os.path.join(ORACLE_DIR, "oracle.c"), "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("gcc failed:\n" + res.stdout + res.stderr)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
