"""Build the gfx950 library ``libcrfinside.so`` in-tree with hipcc."""
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
SOURCES = [os.path.join(CSRC, "crf_kernels.hip"), os.path.join(CSRC, "crf_biaffine.hip"),
           os.path.join(CSRC, "crf_plan.cpp")]
LIB = os.path.join(PKG, "libcrfinside.so")
# microbenchmarks of the ceilings behind the roofline (bench.py --ceilings)
CEIL_SOURCES = [os.path.join(CSRC, "crf_ceilings.hip")]
CEIL_LIB = os.path.join(PKG, "libcrfceilings.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared",
    "--offload-arch=gfx950",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # no NaN ever reaches the charts; lets max fold into v_max_f32_dpp / v_max3
    "-fno-honor-nans",
    # keep single-lane atomics plain: the wave-aggregating rewrite waits for
    # the result at once, which would stall the fused kernel's early claims
    "-mllvm", "-amdgpu-atomic-optimizer-strategy=None",
    "-Wall", "-Wno-unused-function",
    "-I" + os.path.join(ROOT, "include"),
]


def _compile(sources, lib, verbose):
    tmp = lib + ".tmp"
    cmd = [HIPCC, *FLAGS, "-o", tmp, *sources]
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    """Compile every HIP source: ``libcrfinside.so`` (the CRF library) and
    ``libcrfceilings.so`` (ceiling microbenchmarks).  Always recompiles."""
    _compile(SOURCES, LIB, verbose)
    _compile(CEIL_SOURCES, CEIL_LIB, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
