"""Build the gfx950 library ``libcrfinside.so`` in-tree with hipcc."""
import os
import re
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


# Per-kernel register, scratch and LDS use of the last build of LIB (one
# line per kernel, tab-separated, from the compiler's resource remarks).
RESOURCES = os.path.join(PKG, "libcrfinside.resources.tsv")
RESOURCE_FIELDS = ("VGPRs", "AGPRs", "TotalSGPRs", "ScratchSize [bytes/lane]", "VGPRs Spill", "SGPRs Spill",
                   "Occupancy [waves/SIMD]", "LDS Size [bytes/block]")
_REMARK = re.compile(r"remark:\s+(Function Name|" + "|".join(re.escape(f) for f in RESOURCE_FIELDS)
                     + r"):\s+(\S+)\s+\[-Rpass-analysis=kernel-resource-usage\]")


def _demangle(names):
    try:
        out = subprocess.run(["c++filt"], input="\n".join(names), capture_output=True, text=True, check=True)
        dem = out.stdout.split("\n")
        if len(dem) >= len(names):
            return dem[:len(names)]
    except (OSError, subprocess.CalledProcessError):
        pass
    return list(names)


def _write_resources(stderr_text, path):
    rows, cur = [], None
    for line in stderr_text.splitlines():
        m = _REMARK.search(line)
        if not m:
            continue
        if m.group(1) == "Function Name":
            cur = {"name": m.group(2)}
            rows.append(cur)
        elif cur is not None:
            cur[m.group(1)] = m.group(2)
    names = _demangle([r["name"] for r in rows])
    with open(path, "w") as f:
        f.write("\t".join(("kernel", "mangled") + RESOURCE_FIELDS) + "\n")
        for r, d in zip(rows, names):
            f.write("\t".join([d, r["name"]] + [r.get(k, "") for k in RESOURCE_FIELDS]) + "\n")


def _compile(sources, lib, verbose, resources=None):
    tmp = lib + ".tmp"
    cmd = [HIPCC, *FLAGS, "-o", tmp, *sources]
    if resources is not None:
        cmd[1:1] = ["-Rpass-analysis=kernel-resource-usage", "-fno-caret-diagnostics"]
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    if resources is None:
        subprocess.run(cmd, check=True)
    else:
        r = subprocess.run(cmd, capture_output=True, text=True)
        rest = "\n".join(ln for ln in r.stderr.splitlines() if "kernel-resource-usage" not in ln)
        if rest.strip():
            print(rest, file=sys.stderr)
        if r.stdout.strip():
            print(r.stdout, file=sys.stderr)
        if r.returncode != 0:
            raise subprocess.CalledProcessError(r.returncode, cmd)
        _write_resources(r.stderr, resources)
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    """Compile every HIP source: ``libcrfinside.so`` (the CRF library, with
    its kernels' resource report beside it) and ``libcrfceilings.so``
    (ceiling microbenchmarks).  Always recompiles."""
    _compile(SOURCES, LIB, verbose, resources=RESOURCES)
    _compile(CEIL_SOURCES, CEIL_LIB, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
