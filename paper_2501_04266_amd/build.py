"""Build the HIP library libzq.so (gfx950) in-tree, and the benchmark's
bandwidth-ceiling kernels libzq_probe.so.

    python -m paper_2501_04266_amd.build

Flags that matter for exactness: -ffp-contract=off (never fuse a*b+c),
no fast-math, correctly rounded fp32 division/sqrt, fp32 denormals kept.
Packed-fp32 instructions are disabled on purpose.
"""
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libzq.so")
SOURCES = [os.path.join(CSRC, f) for f in ("zq_kernels.hip", "zq_gemm.hip", "zq_api.hip")]
PROBE_LIB = os.path.join(PKG, "libzq_probe.so")
PROBE_SOURCES = [os.path.join(CSRC, "zq_probe.hip")]

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-fast-math",
    "-fhip-fp32-correctly-rounded-divide-sqrt", "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
]


def hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(out=LIB, extra=(), sources=None):
    """Compile every source into `out` (always recompiles)."""
    tmp = out + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, *extra, "-I", INCLUDE, "-I", CSRC, "-o", tmp, *(sources or SOURCES)]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def build_probe(out=PROBE_LIB):
    """The benchmark's bandwidth-ceiling kernels (always recompiles)."""
    return build(out, sources=PROBE_SOURCES)


if __name__ == "__main__":
    print(build())
    print(build_probe())
    sys.exit(0)
