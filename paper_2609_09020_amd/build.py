"""Build the HIP libraries for gfx950 (in-tree).

Every translation unit under csrc/ is compiled by hipcc in parallel into
_build/, then linked into paper_2609_09020_amd/libpic_decode.so (the
decoder).  peaks/k_peaks.hip becomes libpic_peaks.so: the peak-rate
microbenchmarks `bench.py --peaks` runs, not part of the decoder.  Flags:
  -ffp-contract=off          multiplies and adds round exactly as written;
                              fused operations are spelled out as fmaf
  -packed-fp32-ops disabled  no packed fp32 VALU instructions are emitted
  -fvisibility=hidden        only the C ABI (PIC_API) is exported
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libpic_decode.so")
PEAKS_SRC = os.path.join(PKG, "peaks", "k_peaks.hip")
PEAKS_LIB = os.path.join(PKG, "libpic_peaks.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

CFLAGS = ["-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC", "-fvisibility=hidden",
          "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-mllvm", "-amdgpu-mfma-vgpr-form",
          "-Wall", "-Wno-unused-function", "-I", INCLUDE, "-I", CSRC]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC, *CFLAGS, "-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l and l.strip())
    if err and verbose:
        print(err, flush=True)
    return obj


def _link(objs, lib, verbose):
    tmp = lib + f".tmp{os.getpid()}"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, lib)


def build(verbose: bool = False, jobs: int = 8) -> str:
    os.makedirs(BUILD, exist_ok=True)
    # the wide reference-family instances take longest to compile: start them first
    srcs = sorted(sources() + [PEAKS_SRC], key=lambda s: 0 if "_w128" in s or "_w96" in s else 1)
    with cf.ThreadPoolExecutor(max_workers=min(jobs, len(srcs))) as ex:
        objs = dict(zip(srcs, ex.map(lambda s: _compile(s, verbose), srcs)))
    _link([objs[s] for s in sources()], LIB, verbose)
    _link([objs[PEAKS_SRC]], PEAKS_LIB, verbose)
    return LIB


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    print(LIB)
