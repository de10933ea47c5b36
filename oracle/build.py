"""Build the CPU reference library (gcc, OpenMP). TEST INFRASTRUCTURE ONLY."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))


def build(verbose: bool = False) -> str:
    src = os.path.join(HERE, "mcpu_oracle.c")
    out = os.path.join(HERE, "libmcpu_oracle.so")
    # -O2 without -ffast-math: IEEE semantics, no reassociation of the plain loops
    cmd = ["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-std=c11", "-Wall", "-o", out + ".tmp",
           src, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
