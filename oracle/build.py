"""Build step for the float64 CPU oracle (test infrastructure).

Compiles ``nystra_oracle.c`` with gcc into ``libnystra_oracle.so`` next to it.
Generic x86-64 code generation is used on purpose: the library is built in one
container and may be loaded on another host.

With NYSTRA_ORACLE_SANITIZE=1 in the environment the library is built with
AddressSanitizer and UndefinedBehaviorSanitizer instead (any UB report aborts).
A Python process can only load it with gcc's ASan runtime preloaded:

    NYSTRA_ORACLE_SANITIZE=1 python oracle/build.py
    LD_PRELOAD=$(gcc -print-file-name=libasan.so) ASAN_OPTIONS=detect_leaks=0 \\
        python -m pytest tests -m "not gpu"

(leak detection is off: the interpreter itself holds memory until exit).
Rebuild without the variable afterwards.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "nystra_oracle.c")
LIB = os.path.join(HERE, "libnystra_oracle.so")

SANITIZE = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
            "-fno-omit-frame-pointer", "-g"]


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    san = SANITIZE if os.environ.get("NYSTRA_ORACLE_SANITIZE") == "1" else []
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-Wall", "-Wextra",
           "-Werror", *san, SRC, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
