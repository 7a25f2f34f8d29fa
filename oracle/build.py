"""Build the fp64 CPU oracle (test infrastructure) with the host compiler.

The oracle is plain C++17 with no GPU headers; it is compiled with g++ -O2 and
without -ffast-math so that every fp64 operation is the IEEE one written in
the source.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libosd_ref.so")


def build(verbose: bool = False) -> str:
    src = os.path.join(HERE, "osd_ref.cpp")
    cmd = ["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-fno-fast-math", "-ffp-contract=off", "-o", LIB + ".tmp", src]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
