"""Build the CPU oracle (test infrastructure) into oracle/liboracle.so, and
its multi-core variant (oracle.c + oracle_mt.c under OpenMP) into
oracle/liboracle_mt.so.

Plain gcc, IEEE fp32 arithmetic on SSE, no contraction into FMA, no
fast-math, no flush-to-zero.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
SRC_MT = os.path.join(HERE, "oracle_mt.c")
LIB = os.path.join(HERE, "liboracle.so")
LIB_MT = os.path.join(HERE, "liboracle_mt.so")

CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
          "-fno-fast-math", "-mfpmath=sse", "-msse2", "-Wall", "-Wextra"]


def _compile(sources, out, extra, verbose):
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", *CFLAGS, *extra, *sources, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def build(verbose: bool = False) -> str:
    """Compile both libraries; returns the path of the single-threaded one."""
    _compile([SRC], LIB, [], verbose)
    _compile([SRC, SRC_MT], LIB_MT, ["-fopenmp"], verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
