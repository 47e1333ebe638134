"""Build tests/c/abi_round: a plain-C program that drives the library's C ABI
next to the oracle (test code; run by tests/test_gpu_c_abi.py)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
EXE = os.path.join(HERE, "abi_round")


def build():
    pkg = os.path.join(ROOT, "paper_2609_20359_amd")
    orc = os.path.join(ROOT, "oracle")
    rpath = "$ORIGIN/../../paper_2609_20359_amd:$ORIGIN/../../oracle:/opt/rocm/lib"
    subprocess.run(["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
                    "-I/opt/rocm/include", "-I", os.path.join(ROOT, "include"), "-I", orc,
                    "-o", EXE, os.path.join(HERE, "abi_round.c"),
                    "-L", pkg, "-lflround", "-L", orc, "-loracle", "-L/opt/rocm/lib",
                    "-lamdhip64", "-lm", "-Wl,-rpath," + rpath], check=True)
    return EXE


if __name__ == "__main__":
    build()
