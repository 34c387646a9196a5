"""Build the fp64 CPU oracle (test infrastructure only) with gcc.

The oracle is plain C compiled for the host; it never touches the GPU and
shares no source with the HIP library.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "ref_decode.c")
LIB = os.path.join(HERE, "libapex_oracle.so")


def build(extra_flags=(), out=LIB, quiet=False):
    """Compile ref_decode.c into a shared library; returns its path."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
           "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra",
           *extra_flags, SRC, "-o", out + ".tmp", "-lm"]
    if not quiet:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    build()
    sys.exit(0)
