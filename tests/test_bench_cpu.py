"""The benchmark's contract, checked without a GPU: its refusal of more than
one GPU, the algorithmic byte counts it divides by, and the readers of the
committed rocprofv3 and probe summaries it reports from."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from synth import workloads as W  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


@pytest.mark.parametrize("name,per_param", [
    # A (2R + 26) + (2G + 6): a fused local step moves 2R bytes of peer
    # gradients, reads and writes fp32 master/m/v (24) and writes the bf16
    # working copy (2); FedAvg reads G bf16 replicas and writes master and
    # working copy
    ("llama8b_s8", 8 * (2 * 8 + 26) + (2 * 4 + 6)),
    ("hsdp_s4", 8 * (2 * 4 + 26) + (2 * 4 + 6)),
    ("fedavg_heavy", 1 * (2 * 4 + 26) + (2 * 8 + 6)),
    ("stress", 4 * (2 * 16 + 26) + (2 * 16 + 6)),
    # FL+HSDP member: + own wire written (2) and H wire shards read (2H)
    # after the wire pass (2R read + 2 written) ... (2 + 2H) on top of the step
    ("hsdp_s4_h2", 8 * (2 * 4 + 26 + 2 + 2 * 2) + (2 * 4 + 6)),
    # receiver: the broadcast fp32 shard read, master and working written
    ("hsdp_s4_h2_recv", 8 * (2 * 4 + 26 + 2 + 2 * 2) + (4 + 4 + 2)),
    # outer step: + round-start model and momentum buffer read and written
    ("llama8b_s8_outer", 8 * (2 * 8 + 26) + (2 * 4 + 6 + 16)),
    # clipped with the scratch: (2R + 4) then 30
    ("llama8b_s8_clip", 8 * (2 * 8 + 4 + 30) + (2 * 4 + 6)),
])
def test_algorithmic_bytes_per_round(name, per_param):
    w = W.ALL[name]()
    assert w.round_bytes() == w.n * per_param


def test_the_8b_round_moves_350_bytes_per_parameter():
    w = W.llama8b_s8()
    assert w.n == 1_003_782_144 and w.n_seg == 290
    assert w.round_bytes() == 351_323_750_400


BENCH_WORKLOADS = ["tiny", "llama8b_s8", "fedavg_heavy", "hsdp_s4", "stress"]


@pytest.mark.parametrize("name", BENCH_WORKLOADS)
def test_committed_traffic_summary_matches_the_kernel_source(name):
    """Every benchmarked workload has a counter summary for the current
    kernels, and a full-size local step moves close to its algorithmic bytes
    (the 1 Mi-element round stays partly in the caches)."""
    t = bench.read_traffic(name, bench.kernel_source_hash())
    if t is None:
        pytest.skip("the committed traffic summary of %s predates the current kernel source; "
                    "bench.py reports roofline.traffic as null until it is retaken" % name)
    w = W.ALL[name]()
    ratio = t / (w.n * w.step_bytes_per_param())
    if w.n >= 1 << 26:
        assert 0.98 <= ratio < 1.05
    else:
        assert 0.0 < ratio < 1.05


def test_kernel_source_hash_ignores_comments(tmp_path, monkeypatch):
    a = tmp_path / "a.hip"
    a.write_text("int f(int x) { return x + 1; }  // one\n/* block */\n")
    b = tmp_path / "b.hip"
    b.write_text("// header\nint f(int x)  {\n  return x + 1;\n}\n")
    c = tmp_path / "c.hip"
    c.write_text("int f(int x) { return x + 2; }\n")
    hashes = []
    for p in (a, b, c):
        monkeypatch.setattr(bench, "KERNEL_SOURCES", [str(p)])
        hashes.append(bench.kernel_source_hash())
    assert hashes[0] == hashes[1] != hashes[2]


def test_probe_reference_reads_the_committed_summaries():
    pc = bench.probe_reference(W.llama8b_s8(), 5200.0)
    assert pc is not None and 4000 < pc["gbs"] < 8000
    assert pc["frac"] == round(5200.0 / pc["gbs"], 4)
    assert bench.probe_reference(W.hsdp_s4(), 5200.0) is not None
    assert bench.probe_reference(W.stress(), 5200.0) is None   # no probe of that shard


def test_trace_summary_format(tmp_path):
    csv = tmp_path / "stats.csv"
    csv.write_text('"Name","Calls","TotalDurationNs","AverageNs","Percentage","MinNs","MaxNs"\n'
                   '"k_step<8, 0, true>(flr::StepArgs)",8,64000000,8000000.0,90.0,7900000,8100000\n')
    out = bench.summarize_trace(str(csv), "cmd", "llama8b_s8")
    assert "llama31_8b_fsdp_s8_r8_g4_a8" in out
    assert "| k_step<8, 0, true>(flr::StepArgs) | 8 | 8000.0 | 7900.0 | 8100.0 | 90.00 % |" in out


def test_cpu_baseline_runs_the_oracle_on_host_threads():
    cb = bench.cpu_baseline(W.llama8b_s8(), 1 << 16, min_seconds=0.5, n_one=1 << 15)
    assert cb["kind"] == "oracle" and cb["unit"] == "GB/s"
    assert cb["rounds"] >= 1 and cb["seconds"] >= 0.5
    assert cb["cores"] >= 1 and cb["value"] > 0 and cb["one_thread_gbs"] > 0
    assert "%d elements" % (1 << 16) in cb["sample"]
    assert cb["one_thread_elements"] == 1 << 15


def test_live_probe_parsing_and_patterns():
    table = ("| pattern | stores | 1/CU | best | of peak |\n|---|---|---|---|---|\n"
             "| step_R8   | plain |  5286.4 |  5286.4 (1/CU) |  66.1 % |\n"
             "| step_R8   | nt    |  5307.7 |  5307.7 (1/CU) |  66.3 % |\n"
             "| step_R8_w | nt    |  4982.6 |  4982.6 (1/CU) |  62.3 % |\n")
    assert bench.parse_probe_rate(table, "step_R8") == 5307.7
    assert bench.parse_probe_rate(table, "step_R8_w") == 4982.6
    assert bench.parse_probe_rate(table, "step_R4") is None
    assert bench.step_pattern(W.llama8b_s8()) == "step_R8"
    assert bench.step_pattern(W.hsdp_s4()) == "step_R4"
    assert bench.step_pattern(W.stress()) is None                  # R = 16: no such pattern
    assert bench.step_pattern(W.llama8b_s8_clip()) is None         # clipped: two passes
    assert bench.step_pattern(W.hsdp_s4_h2()) is None              # FL+HSDP: wire + tier 2


def test_every_placement_choice_names_an_exported_function():
    """bench.py --placement resolves each choice to a function the package
    exports (None: torch's allocator); the default is the staggered pool."""
    import paper_2609_20359_amd as P

    assert set(bench.PLACEMENTS) == {"staggered", "separate", "torch"}
    for name, (fn, label) in bench.PLACEMENTS.items():
        assert label
        assert fn is None or callable(getattr(P, fn)), name
    assert bench.PLACEMENTS["staggered"][0] == "place_arrays"
