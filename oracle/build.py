"""Build the CPU oracle library (oracle/libeao.so) with gcc.

The oracle is test infrastructure: the product library never links or loads
it.  `python oracle/build.py` or `oracle.build.build()` compiles it in place.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCES = ["eao.c", "eao_tier.c", "eao_stack.c"]
LIB = os.path.join(HERE, "libeao.so")


def build(verbose: bool = False) -> str:
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-Werror", "-fPIC",
           "-shared", "-o", LIB + ".tmp"] + [os.path.join(HERE, s) for s in SOURCES]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
