"""Builds the synthetic-input library ``libsynth.so``."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))


# The sanitizer build (AddressSanitizer and UndefinedBehaviorSanitizer, every
# finding fatal) that the CPU test tier runs the oracle's pins against.
SANITIZE = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
            "-fno-sanitize-recover=all"]


def build(verbose=False, out=None, sanitize=False):
    out = out or os.path.join(HERE, "libsynth.so")
    opt = SANITIZE if sanitize else ["-O3"]
    cmd = ["g++", *opt, "-std=c++17", "-shared", "-fPIC", "-pthread", "-Wall",
           os.path.join(HERE, "synth.cpp"), "-o", out]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return out


if __name__ == "__main__":
    build(verbose=True)
