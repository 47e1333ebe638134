"""The C ABI from plain C: tests/c/abi_round (built by __graft_entry__.build())
runs one fl_round on hipMalloc'd buffers and compares it bit for bit with the
oracle, with no Python or torch in the process."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c", "abi_round")


def test_fl_round_from_plain_c():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    assert os.path.exists(EXE), "%s is not built; run __graft_entry__.build()" % EXE
    print("[gpu-c-abi] running", EXE, flush=True)
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, r.stderr
    assert "abi_round ok" in r.stdout
