"""Build the synthetic-input generator libraries in place.

libsynth_host.so  -- gcc build of synth_host.c (host values, sampled gathers)
libsynth_dev.so   -- hipcc build of synth_dev.hip for gfx950 (HBM fills)

Both are compiled with -ffp-contract=off: the generator relies on the two
builds producing identical bits for every (seed, stream, index).
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

HOST_LIB = os.path.join(HERE, "libsynth_host.so")
DEV_LIB = os.path.join(HERE, "libsynth_dev.so")


def _run(cmd):
    subprocess.run(cmd, check=True, cwd=HERE)


def build_host():
    _run(["gcc", "-std=c11", "-O2", "-fPIC", "-shared", "-ffp-contract=off",
          "-fno-fast-math", "-Wall", "-Wextra", "-o", HOST_LIB, "synth_host.c", "-lpthread"])


def build_dev():
    _run([HIPCC, "--offload-arch=gfx950", "-O3", "-fPIC", "-shared",
          "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wno-unused-command-line-argument", "-o", DEV_LIB, "synth_dev.hip"])


def build():
    build_host()
    build_dev()


if __name__ == "__main__":
    build()
