"""bench.py end to end on the GPU, on the small workload: the JSON line of the
contract for each placement of the shard's arrays, with the live probe and a
short oracle leg on the default placement."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _bench(*args):
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "tiny", "--steps", "3",
           "--warmup", "1"] + list(args)
    print("[gpu-bench]", " ".join(cmd[1:]), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, r.stdout
    return json.loads(lines[0])


@pytest.mark.parametrize("placement,name", [("separate", "one exact-size hipMalloc per array"),
                                            ("torch", "torch's caching allocator")])
def test_bench_line_for_each_placement(gpu, placement, name):
    d = _bench("--no-cpu", "--no-probe", "--placement", placement)
    assert d["config"]["placement"] == name
    assert d["config"]["workload"] == "tiny_n1m_r4_g2_a4"
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1
    assert d["value"] > 0 and d["ms_per_step"] > 0 and d["cpu_baseline"] is None
    r = d["roofline"]
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert r["achieved"] > 0 and abs(r["frac"] - r["achieved"] / r["peak"]) < 1e-3


def test_bench_line_default_placement_with_probe_and_oracle(gpu):
    d = _bench("--cpu-seconds", "0.5")
    assert d["config"]["placement"].startswith("one pool")
    live = d["roofline"].get("probe_live")
    assert live is not None and live["stagger_bytes"] == 2048 and live["gbs"] > 0
    c = d["cpu_baseline"]
    assert c["kind"] == "oracle" and c["value"] > 0 and c["cores"] >= 1 and c["sample"]
