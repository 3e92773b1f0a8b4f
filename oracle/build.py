"""Build step for the float64 CPU oracle (test infrastructure).

Compiles ``nystra_oracle.c`` with gcc into ``libnystra_oracle.so`` next to it.
Generic x86-64 code generation is used on purpose: the library is built in one
container and may be loaded on another host.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "nystra_oracle.c")
LIB = os.path.join(HERE, "libnystra_oracle.so")


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-Wall", "-Wextra",
           "-Werror", SRC, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
