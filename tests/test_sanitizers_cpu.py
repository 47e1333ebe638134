"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer, built into
a temporary directory and exercised in a child process, so that an
out-of-bounds access, a use after free or an undefined operation (signed
overflow, a bad shift, a misaligned load) aborts the child and fails the
test:
  * the oracle (oracle/oracle.c) and the host build of the input generator
    (synth/synth_host.c), built with gcc, under the oracle's pins and the
    whole-shard sampling tests;
  * the C-ABI layer's host code (the library built with the sanitizers on
    its host side only), under the ABI tests that run without a GPU:
    argument validation, fingerprints, the layout table build, the
    learning-rate schedule."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
       "-fno-sanitize-recover=undefined"]
COMMON = ["-std=c11", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math", "-Wall"]


HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _runtime(gcc, name):
    path = subprocess.run([gcc, "-print-file-name=" + name], capture_output=True, text=True,
                          check=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_oracle_and_generator_under_asan_and_ubsan(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not found")
    asan = _runtime(gcc, "libasan.so")
    if asan is None:
        pytest.skip("gcc's AddressSanitizer runtime not found")
    ora = str(tmp_path / "liboracle_san.so")
    gen = str(tmp_path / "libsynth_host_san.so")
    subprocess.run([gcc] + COMMON + SAN + ["-I", os.path.join(ROOT, "oracle"), "-o", ora,
                                           os.path.join(ROOT, "oracle", "oracle.c"), "-lm"],
                   check=True)
    subprocess.run([gcc] + COMMON + SAN + ["-o", gen, os.path.join(ROOT, "synth", "synth_host.c"),
                                           "-lpthread"], check=True)
    for lib in (ora, gen):
        with open(lib, "rb") as f:
            assert b"__asan_report" in f.read()
    env = dict(os.environ)
    env["ORACLE_LIB"] = ora
    env["SYNTH_HOST_LIB"] = gen
    # the ASan runtime must come first among the preloaded libraries of the
    # (uninstrumented) Python process; anything already preloaded stays
    env["LD_PRELOAD"] = asan + (":" + env["LD_PRELOAD"] if env.get("LD_PRELOAD") else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    probe = subprocess.run([sys.executable, "-c",
                            "import oracle, synth; oracle.lib(); synth.host_lib(); "
                            "print(oracle._LIB_PATH)"],
                           env=env, cwd=ROOT, capture_output=True, text=True, timeout=300)
    assert probe.returncode == 0, probe.stderr[-4000:]
    assert probe.stdout.strip() == ora
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-m", "not gpu",
                        "-p", "no:cacheprovider", "tests/test_oracle_pins.py",
                        "tests/test_sampling_cpu.py"],
                       env=env, cwd=ROOT, capture_output=True, text=True, timeout=1200)
    assert r.returncode == 0, (r.stdout[-4000:], r.stderr[-4000:])
    assert " passed" in r.stdout


def _clang_asan_runtime():
    r = subprocess.run([HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"],
                       capture_output=True, text=True)
    path = r.stdout.strip()
    if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path):
        return path
    import glob

    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


def test_abi_host_code_under_asan_and_ubsan(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not found")
    asan = _clang_asan_runtime()
    if asan is None:
        pytest.skip("clang's AddressSanitizer runtime not found")
    from paper_2609_20359_amd import build as B

    out = str(tmp_path / "libflround_san.so")
    host_san = []
    for f in ("-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
              "-fno-omit-frame-pointer"):
        host_san += ["-Xarch_host", f]
    B.build(out=out, extra=host_san + ["-Xarch_host", "-g"])
    with open(out, "rb") as f:
        assert b"__asan_report" in f.read()   # the host code is instrumented
    env = dict(os.environ)
    env["FLROUND_LIB"] = out
    env["LD_PRELOAD"] = asan + (":" + env["LD_PRELOAD"] if env.get("LD_PRELOAD") else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-m", "not gpu",
                        "-p", "no:cacheprovider", "tests/test_abi_cpu.py"],
                       env=env, cwd=ROOT, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, (r.stdout[-4000:], r.stderr[-4000:])
    assert " passed" in r.stdout
