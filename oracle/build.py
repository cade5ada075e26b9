"""Build the oracle's shared library (test infrastructure only).

The oracle is compiled with gcc, without fast-math and without floating-point
contraction, so each entry is the plain ascending-k fp64 sum. OpenMP is used
when the compiler supports it (it only splits rows between threads).
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "gemm_ref.c")
LIB = os.path.join(HERE, "libgemm_ref.so")


def build(out=LIB, extra_defines=()):
    """Compile gemm_ref.c into `out`. `extra_defines` is for tests only."""
    base = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-std=c11",
            "-shared", "-fPIC", SRC, "-o", out + ".tmp"]
    base += ["-D%s" % d for d in extra_defines]
    cmd = base[:1] + ["-fopenmp"] + base[1:] + ["-lm"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:  # no OpenMP runtime: build single-threaded
        r = subprocess.run(base + ["-lm"], capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("oracle build failed:\n" + r.stderr)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(*sys.argv[1:2]))
