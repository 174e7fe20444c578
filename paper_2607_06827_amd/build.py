"""Build libspeechkv.so for gfx950 with hipcc, in-tree.

    python -m paper_2607_06827_amd.build

Every HIP source under csrc/ is compiled to an object in _build/ and linked
into paper_2607_06827_amd/libspeechkv.so; the benchmark's streaming-read
ceiling kernel (csrc_bench/) goes into its own libskv_bench.so, which only
bench.py loads.  Packed fp32 instructions are disabled for every device
compile.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
CSRC_BENCH = os.path.join(HERE, "csrc_bench")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libspeechkv.so")
BENCH_LIB = os.path.join(HERE, "libskv_bench.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

DEVICE_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # keep MFMA accumulators in ordinary VGPRs: the softmax rescales them with
    # VALU ops, and AGPR accumulators cost a copy each way every tile
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-Wall", "-Wno-unused-function",
]


def _compile_and_link(sources, lib, verbose):
    procs = []
    objs = []
    for src in sources:
        obj = os.path.join(BUILD, os.path.basename(src) + ".o")
        objs.append(obj)
        cmd = [HIPCC, *DEVICE_FLAGS, "-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                                            text=True)))
    failed = []
    for src, p in procs:
        out, _ = p.communicate()
        # the host pass does not know the packed-fp32 feature and says so; keep
        # every other line
        lines = [l for l in out.splitlines() if "packed-fp32-ops" not in l]
        if lines and (verbose or p.returncode):
            print("\n".join(lines), file=sys.stderr)
        if p.returncode:
            failed.append(src)
    if failed:
        raise RuntimeError(f"hipcc failed for {failed}")
    tmp = lib + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    """Compile every csrc/*.hip and link libspeechkv.so, then the benchmark's
    libskv_bench.so.  Returns the path of libspeechkv.so."""
    os.makedirs(BUILD, exist_ok=True)
    _compile_and_link(sorted(glob.glob(os.path.join(CSRC, "*.hip"))), LIB, verbose)
    _compile_and_link(sorted(glob.glob(os.path.join(CSRC_BENCH, "*.hip"))), BENCH_LIB, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
