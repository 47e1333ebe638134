"""Build libflround.so (the C-ABI library and its gfx950 kernels) in place.

    python -m paper_2609_20359_amd.build

Flags: -O3 for gfx950 only; -ffp-contract=off so that no multiply and add
are fused (every fp32 operation of the method is rounded on its own);
packed-fp32 instructions disabled.  HIP's default correctly rounded fp32
division and square root, and its default of keeping subnormals, are left
on.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
LIB = os.path.join(HERE, "libflround.so")
SOURCES = [os.path.join(HERE, "csrc", "flround_api.cpp"),
           os.path.join(HERE, "csrc", "flround_kernels.hip")]

HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Wall", "-Wno-unused-command-line-argument"]


def build(out=LIB, extra=()):
    cmd = [HIPCC] + HIP_FLAGS + list(extra) + ["-shared", "-I", os.path.join(ROOT, "include"),
                                               "-I", os.path.join(HERE, "csrc"), "-o", out] + SOURCES
    subprocess.run(cmd, check=True)
    return out


if __name__ == "__main__":
    build()
