"""Compile libsynth.so from synth.c with gcc (host code only)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
FLAGS = ["-O3", "-mavx2", "-ffp-contract=off", "-fno-math-errno", "-fno-trapping-math",
         "-fopenmp", "-Wall", "-shared", "-fPIC"]


def build(verbose=False):
    src = os.path.join(HERE, "synth.c")
    out = os.path.join(HERE, "libsynth.so")
    tmp = out + ".tmp"
    cmd = ["gcc", *FLAGS, src, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    build(verbose=True)
