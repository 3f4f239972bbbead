"""Build the CPU oracle (plain C, gcc) into oracle/libpic_oracle.so.

Test infrastructure: the oracle is what the decoder's results are checked
against.  ``-ffp-contract=off`` keeps every multiply and add of the fp64 and
fp32 models rounded exactly as written in the source.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "pic_oracle.c")
ZPR_SRC = os.path.join(HERE, "zpr_oracle.c")
HUFF_SRC = os.path.join(HERE, "huff_oracle.c")
SRCS = (SRC, ZPR_SRC, HUFF_SRC)
LIB = os.path.join(HERE, "libpic_oracle.so")


def build(verbose: bool = False, srcs=SRCS, out: str = LIB, extra_flags=()) -> str:
    """Compile the C files ``srcs`` (default: the oracle's) into the shared
    library ``out``; ``extra_flags`` go to gcc as well (e.g. sanitizers)."""
    tmp = out + f".tmp{os.getpid()}"
    cmd = ["gcc", "-O2", "-std=c99", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-Wall", "-Wextra", *extra_flags, "-o", tmp, *srcs, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
