"""Compile tests/c/abi_check.c (a plain C11 consumer of include/zq.h, linked
with libzq.so and the CPU oracle) -- test infrastructure."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "abi_check.c")
ORACLE = os.path.join(ROOT, "oracle", "zq_oracle.c")
PKG = os.path.join(ROOT, "paper_2501_04266_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def flags():
    return ["-std=c11", "-Wall", "-Wextra", "-Werror", "-pedantic", "-O2", "-fno-fast-math", "-ffp-contract=off",
            "-fopenmp", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
            "-isystem", os.path.join(ROCM, "include")]


def syntax_check():
    """include/zq.h alone compiles as strict C99 and C11, and the consumer
    compiles as strict C11 (the HIP runtime headers as system headers)."""
    for std in ("-std=c99", "-std=c11"):
        subprocess.run(["gcc", std, "-Wall", "-Wextra", "-Werror", "-pedantic", "-fsyntax-only", "-x", "c",
                        "-I", os.path.join(ROOT, "include"), "-"], input=b'#include "zq.h"\n', check=True)
    subprocess.run(["gcc", *flags(), "-fsyntax-only", SRC], check=True)


def build(out=None):
    out = out or os.path.join(HERE, "abi_check")
    cmd = ["gcc", *flags(), "-o", out, SRC, ORACLE, "-L", PKG, "-lzq", "-L", os.path.join(ROCM, "lib"),
           "-lamdhip64", "-Wl,-rpath," + PKG, "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-lm", "-lgomp"]
    subprocess.run(cmd, check=True)
    return out
