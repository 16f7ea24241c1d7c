"""Builds the CPU oracle library ``libggref.so`` (test infrastructure)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))


def build(verbose=False):
    out = os.path.join(HERE, "libggref.so")
    cmd = ["g++", "-O3", "-std=c++17", "-ffp-contract=off", "-shared", "-fPIC", "-Wall", "-Wextra",
           os.path.join(HERE, "ggref.cpp"), "-o", out]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return out


if __name__ == "__main__":
    build(verbose=True)
