"""Builds the oracle's C helper (wgen.c -> liboracle.so) with gcc.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SO_PATH = os.path.join(HERE, "liboracle.so")


def build(verbose: bool = False) -> str:
    src = os.path.join(HERE, "wgen.c")
    tmp = SO_PATH + ".tmp"
    cmd = ["gcc", "-O3", "-fopenmp", "-shared", "-fPIC", "-std=c11", src, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, SO_PATH)
    return SO_PATH


if __name__ == "__main__":
    print(build(verbose=True))
