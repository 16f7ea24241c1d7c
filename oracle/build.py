"""Builds the CPU oracle library ``libggref.so`` (test infrastructure)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))


# The sanitizer build (AddressSanitizer and UndefinedBehaviorSanitizer, every
# finding fatal) that the CPU test tier runs the oracle's pins against.
SANITIZE = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
            "-fno-sanitize-recover=all"]


def build(verbose=False, out=None, sanitize=False):
    out = out or os.path.join(HERE, "libggref.so")
    opt = SANITIZE if sanitize else ["-O3"]
    cmd = ["g++", *opt, "-std=c++17", "-ffp-contract=off", "-shared", "-fPIC", "-Wall", "-Wextra",
           os.path.join(HERE, "ggref.cpp"), "-o", out]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return out


if __name__ == "__main__":
    build(verbose=True)
