"""Compile the serial CPU oracle (oracle.c) into oracle/liboracle.so with gcc.

Test infrastructure only: the product library never links this file.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")


def compile_source(src: str, out: str, verbose: bool = False) -> str:
    """Compile one oracle source file into a shared library at ``out``."""
    tmp = out + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra", "-Werror",
           "-I", HERE, "-o", tmp, src, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def build(verbose: bool = False) -> str:
    """Always recompiles oracle.c; returns the path of the shared library."""
    return compile_source(SRC, LIB, verbose)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
