"""Build the float64 CPU oracle, ``liblpv_oracle.so`` (test infrastructure).

Plain gcc, no GPU code.  ``-ffp-contract=off`` keeps every multiply and add a
separately rounded float64 operation, so the oracle's result does not depend
on whether the host compiler would fuse them.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liblpv_oracle.so")


def build(verbose: bool = False) -> str:
    src = os.path.join(HERE, "lpv_oracle.c")
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-Wall",
           "-Wextra", "-fPIC", "-shared", "-pthread", src, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
