"""Build the HBM ceiling probe executable (hbmprobe/hbm_probe) for gfx950."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
EXE = os.path.join(HERE, "hbm_probe")


def build():
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-x", "hip",
                    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                    "-Wno-unused-command-line-argument", "-o", EXE,
                    os.path.join(HERE, "hbm_probe.cpp")], check=True)
    return EXE


if __name__ == "__main__":
    build()
