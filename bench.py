"""Benchmark of one GPU's share of the FL+FSDP parameter sync (fl_round).

A step is one fl_round: A = 8 fused local steps (R = 8 peer gradients ->
AdamW on the fp32 master shard -> bf16 working copy, with the per-segment
sums of squares of each step's reduced gradient) and one FedAvg of G = 4
federation-group replicas, on the Llama-3.1-8B shard of a rank in a sharding
group of 8 (N = 1,003,782,144 parameters in 290 segments), with every input
already resident in HBM.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu]
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "effective HBM GB/s (% of MI355X peak) and params/s per fl_round, 8B-shaped shard"
PEAK_HBM_GBS = 8000.0   # MI355X HBM3E, 8 TB/s
# --placement: the function of paper_2609_20359_amd that allocates the shard's
# arrays (None: torch's caching allocator) and how the config names it
PLACEMENTS = {
    "staggered": ("place_arrays", "one pool, array k at 2 MiB + k x 2 KiB"),
    "separate": ("separate_arrays", "one exact-size hipMalloc per array"),
    "torch": (None, "torch's caching allocator"),
}
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2609_20359_amd", "csrc", f)
                  for f in ("flround_kernels.hip", "flr_internal.h")]


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def kernel_source_hash():
    """Hash of the kernel sources with comments and whitespace removed, so
    that it changes with the code the counters measured and not with its
    commentary."""
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(p) as f:
            src = f.read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update(" ".join(src.split()).encode())
    return h.hexdigest()[:16]


def read_traffic(workload, current_hash):
    """Counter-measured HBM bytes of one local step of the workload (from the
    rocprofv3 --pmc summary committed under profiles/), or None if there is
    none or the kernel source changed since it was taken."""
    path = traffic_file(workload)
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    fields = dict(re.findall(r"^- (\w+): (\S+)$", txt, flags=re.M))
    if fields.get("kernel_source_hash") != current_hash:
        return None
    try:
        return float(fields["hbm_bytes_per_local_step"])
    except (KeyError, ValueError):
        return None


COPY_KERNEL = "__amd_rocclr_copyBuffer"


def _rt(k):
    """Template count of a dispatched kernel (the generic instance is 0)."""
    return k if k in (1, 2, 4, 8, 16) else 0


def round_kernels(w):
    """(kernel name, algorithmic bytes read, bytes written) per launch for each
    streaming kernel a round of workload w launches (bench.py asks for the
    per-segment sums in every round)."""
    n = w.n
    ks = []
    r = w.H if w.H > 1 else w.R
    if w.H > 1:
        wire = "k_wire<%d>" % w.R if _rt(w.R) else "k_step<0, 3, false>"
        ks.append((wire, 2 * w.R * n, 2 * n))
    if w.max_grad_norm > 0 and w.H == 1 and w.clip_scratch:
        ks.append(("k_step<%d, 1, true>" % _rt(w.R), 2 * w.R * n, 4 * n))
        ks.append(("k_step<1, 2, false>", 16 * n, 14 * n))
    elif w.max_grad_norm > 0:
        ks.append(("k_step<%d, 4, true>" % _rt(r), 2 * r * n, 0))
        ks.append(("k_step<%d, 0, false>" % _rt(r), (2 * r + 12) * n, 14 * n))
    else:
        ks.append(("k_step<%d, 0, true>" % _rt(r), (2 * r + 12) * n, 14 * n))
    if w.H > 1 and not w.hsdp_member:
        ks.append(("k_bcast_recv", 4 * n, 6 * n))
    elif w.outer is not None:
        ks.append(("k_fedavg<%d, true>" % _rt(w.G), (2 * w.G + 8) * n, 14 * n))
    else:
        ks.append(("k_fedavg<%d, false>" % _rt(w.G), 2 * w.G * n, 6 * n))
    return ks


def traffic_file(workload):
    return os.path.join(ROOT, "profiles", "traffic_%s.md" % W_ALL()[workload]().name)


def _pmc_means(path):
    """Per-kernel mean and count of a rocprofv3 --pmc counter_collection CSV."""
    import csv

    acc = {}
    for r in csv.DictReader(open(path)):
        key = (r["Kernel_Name"], int(r["Grid_Size"]))
        acc.setdefault(key, []).append(float(r["Counter_Value"]))
    return {k: (sum(v) / len(v), len(v)) for k, v in acc.items()}


def summarize_pmc(fetch_csv, write_csv, copy_mib, cmd_fetch, cmd_write, workload="llama8b_s8"):
    """Markdown summary of two counter passes (FETCH_SIZE, WRITE_SIZE, KiB per
    dispatch), scaled by what each counter reads for the plain copy of
    copy_mib MiB that the same runs performed, for every streaming kernel a
    round of the workload launches."""
    w = W_ALL()[workload]()
    fetch, write = _pmc_means(fetch_csv), _pmc_means(write_csv)

    def pick(table, name):
        """Mean and count over every dispatch of the kernel (all grid sizes:
        a pass that carries the previous finalize has one more workgroup)."""
        hits = [v for (k, g), v in table.items() if name in k]
        if not hits:
            raise KeyError(name)
        cnt = sum(c for _, c in hits)
        return sum(m * c for m, c in hits) / cnt, cnt

    copy_kib = copy_mib * 1024.0
    cands = [(k, g) for (k, g) in fetch if COPY_KERNEL in k]
    big = max(cands, key=lambda kg: fetch[kg][0])
    f_copy, w_copy = fetch[big][0], write[big][0]
    f_scale, w_scale = copy_kib / f_copy, copy_kib / w_copy
    d = w.describe()
    lines = ["# HBM traffic of the kernels of one round: %s" % d["workload"], "",
             ", ".join("%s=%s" % (k, d[k]) for k in d if k != "workload"), "",
             "Counter passes (one counter per run, KiB per dispatch):", "",
             "    " + cmd_fetch, "    " + cmd_write, "",
             "Calibration: the same runs copy %d MiB with %s (reads and writes %d KiB)." % (
                 copy_mib, COPY_KERNEL, copy_kib),
             "FETCH_SIZE reads %.1f KiB for it -> scale %.5f; WRITE_SIZE reads %.1f KiB -> "
             "scale %.5f." % (f_copy, f_scale, w_copy, w_scale), "",
             "| kernel | dispatches | FETCH_SIZE KiB | WRITE_SIZE KiB | scaled read GB | "
             "scaled write GB | algorithmic read GB | algorithmic write GB | traffic / algorithmic |",
             "|---|---|---|---|---|---|---|---|---|"]
    out = {}
    kernels = round_kernels(w)
    for name, alg_r, alg_w in kernels:
        f, cnt = pick(fetch, name)
        wr, _ = pick(write, name)
        rb, wb = f * f_scale * 1024, wr * w_scale * 1024
        out[name] = rb + wb
        lines.append("| %s | %d | %.1f | %.1f | %.4f | %.4f | %.4f | %.4f | %.4f |" % (
            name, cnt, f, wr, rb / 1e9, wb / 1e9, alg_r / 1e9, alg_w / 1e9,
            (rb + wb) / (alg_r + alg_w)))
    step = kernels[:-1]
    lines += ["", "Values read by bench.py (roofline.traffic: the HBM bytes of one local step, "
              "the kernels %s):" % ", ".join(k for k, _, _ in step), "",
              "- kernel_source_hash: %s" % kernel_source_hash(),
              "- hbm_bytes_per_local_step: %.0f" % sum(out[k] for k, _, _ in step), ""]
    return "\n".join(lines)


def summarize_trace(stats_csv, cmd, workload="llama8b_s8"):
    import csv

    rows = list(csv.DictReader(open(stats_csv)))
    d = W_ALL()[workload]().describe()
    shape = ", ".join("%s=%s" % (k, d[k]) for k in d if k != "workload")
    lines = ["# Kernel trace, one fl_round per step: %s" % d["workload"], "", shape, "",
             "    " + cmd, "",
             "| kernel | calls | average us | min us | max us | share of GPU time |",
             "|---|---|---|---|---|---|"]
    for r in rows:
        lines.append("| %s | %s | %.1f | %.1f | %.1f | %.2f %% |" % (
            r["Name"].replace("|", "/"), r["Calls"], float(r["AverageNs"]) / 1e3,
            float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3, float(r["Percentage"])))
    lines.append("")
    return "\n".join(lines)


PROBE_FILES = {1003782144: os.path.join(ROOT, "profiles", "hbm_probe_reference_llama31_8b_s8.md"),
               2007564288: os.path.join(ROOT, "profiles", "hbm_probe_reference_llama31_8b_s4.md")}


def probe_reference(w, achieved):
    """The rate of the local step's access pattern with no arithmetic, in the
    library's loop and launch structure (a same-design reference, not a
    bound), from the committed probe summary for this shard length, where the
    probe measured the pattern (a plain fused step: one replica, no
    clipping); else None."""
    path = PROBE_FILES.get(w.n)
    pattern = "step_R%d" % w.R
    if not (w.H == 1 and w.max_grad_norm <= 0) or path is None or not os.path.exists(path):
        return None
    best = None
    for line in open(path):
        cells = [c.strip() for c in line.strip().strip("|").split("|")]
        if cells and cells[0] == pattern:
            for c in cells:
                if c.endswith("/CU)"):
                    val = float(c.split()[0])
                    best = val if best is None else max(best, val)
    if best is None:
        return None
    return {"pattern": "%s (%d bf16 streams read, 3 fp32 read and written, 1 bf16 written; "
                       "no arithmetic)" % (pattern, w.R), "gbs": best,
            "frac": round(achieved / best, 4)}


PROBE_EXE = os.path.join(ROOT, "hbmprobe", "hbm_probe")


def step_pattern(w):
    """The probe pattern of the workload's local step (a plain fused step
    with R in {2, 4, 8}: one replica, no clipping), or None."""
    if w.H == 1 and w.max_grad_norm <= 0 and w.R in (2, 4, 8):
        return "step_R%d" % w.R
    return None


def probe_live(w, achieved, stagger, timeout=180):
    """The same-design reference measured on this machine, now: hbm_probe (a
    child process) moves the local step's access pattern over w.n elements
    at one workgroup per CU with no arithmetic, its streams placed as the
    benchmark placed the shard's arrays (stagger bytes; 0: one exact-size
    allocation each).  Returns the pattern, its rate with nontemporal stores and the
    fraction of it the kernel reached, or None when there is no pattern or
    probe."""
    import subprocess

    pattern = step_pattern(w)
    if pattern is None or not os.path.exists(PROBE_EXE):
        return None
    r = subprocess.run([PROBE_EXE, str(w.n), pattern, "1", str(stagger)], capture_output=True,
                       text=True, timeout=timeout)
    if r.returncode != 0:
        log("live probe failed (%d): %s" % (r.returncode, r.stdout[-300:] + r.stderr[-300:]))
        return None
    gbs = parse_probe_rate(r.stdout, pattern)
    if gbs is None:
        return None
    return {"pattern": pattern, "gbs": gbs, "frac": round(achieved / gbs, 4),
            "workgroups_per_cu": 1, "stagger_bytes": stagger}


def parse_probe_rate(text, pattern):
    """GB/s of `pattern` with nontemporal stores at the first workgroups-per-CU
    column of an hbm_probe table, or None."""
    for line in text.splitlines():
        cells = [c.strip() for c in line.strip().strip("|").split("|")]
        if len(cells) >= 4 and cells[0] == pattern and cells[1] == "nt":
            try:
                return float(cells[2])
            except ValueError:
                return None
    return None


def step_label(w):
    """The kernels of one local step, as the roofline figure counts them."""
    fused = "k_step<%s=%d, fused, %s>" % ("R" if w.H == 1 else "H", w.R if w.H == 1 else w.H,
                                         "clipped" if w.max_grad_norm > 0 else
                                         "per-segment sums")
    parts = []
    if w.H > 1:
        parts.append("k_wire<R=%d>" % w.R)
    if w.max_grad_norm > 0:
        parts.append("k_step<%s=%d, sum of squares> + finalize" % (
            "R" if w.H == 1 else "H", w.R if w.H == 1 else w.H))
    parts.append(fused)
    return "one local step: " + " + ".join(parts)


def W_ALL():
    from synth import workloads as W

    return W.ALL


def cpu_baseline(w, n_sample, min_seconds=10.0, max_rounds=10000, n_one=16 << 20):
    """The oracle as it stands, timed on the host's cores: rounds on the first
    n_sample elements of the same shard (same generator, same segments),
    split into one contiguous chunk per thread; every thread runs the
    unchanged single-threaded oracle on its chunk (ctypes releases the GIL).
    Rounds are repeated on the evolving state until min_seconds have passed,
    so that the rate is taken over several seconds of CPU work.  Also the
    one-thread rate of one round on the first n_one elements."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle
    import synth.buffers as B
    from synth import host_threads

    orc = oracle.Oracle()
    n_sample = min(n_sample, w.n)
    T = max(1, min(host_threads(), n_sample))
    bounds = np.linspace(0, n_sample, T + 1).astype(np.int64)
    jobs = []
    for t in range(T):
        lo, hi = int(bounds[t]), int(bounds[t + 1])
        off, dec, _ = w.span_layout(lo, hi)
        jobs.append((B.HostInputs(w, span=(lo, hi)), off, dec))

    def run(job):
        host, off, dec = job
        oracle.workload_round(orc, w, host, seg_off=off, seg_decay=dec, want_sumsq=True)

    per_param = w.A * w.step_bytes_per_param() + w.fedavg_bytes_per_param()
    # one thread, one round, on a slice of up to 16 Mi elements
    n1 = min(n_one, n_sample)
    off1, dec1, _ = w.span_layout(0, n1)
    one = (B.HostInputs(w, span=(0, n1)), off1, dec1)   # inputs generated before the clock
    t0 = time.perf_counter()
    run(one)
    dt1 = time.perf_counter() - t0
    del one
    rounds = 0
    with ThreadPoolExecutor(T) as ex:
        t0 = time.perf_counter()
        while True:
            list(ex.map(run, jobs))
            rounds += 1
            dt = time.perf_counter() - t0
            if dt >= min_seconds or rounds >= max_rounds:
                break
    return dict(value=round(rounds * n_sample * per_param / dt / 1e9, 4), unit="GB/s", cores=T,
                kind="oracle", params_per_s=round(rounds * n_sample / dt, 1),
                seconds=round(dt, 3), rounds=rounds,
                one_thread_gbs=round(n1 * per_param / dt1 / 1e9, 4), one_thread_elements=n1,
                sample="%d rounds with per-segment sums (A=%d, R=%d, G=%d, H=%d) on the first "
                       "%d elements of the same shard, as %d contiguous chunks run concurrently, "
                       "one thread each, by the single-threaded C oracle" % (
                           rounds, w.A, w.R, w.G, w.H, n_sample, T))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama8b_s8")
    ap.add_argument("--cpu-sample", type=int, default=64 << 20)
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="the oracle leg repeats rounds on its sample for at least this long")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--placement", choices=sorted(PLACEMENTS), default="staggered",
                    help="how the shard's arrays are allocated (paper_2609_20359_amd.arena): "
                    "one staggered pool, separate exact-size hipMallocs, or torch's allocator")
    ap.add_argument("--no-probe", action="store_true",
                    help="skip the live same-design reference (hbm_probe) after the timed region")
    ap.add_argument("--blocks-per-cu", type=int, default=0,
                    help="workgroups per CU for every kernel (0: the library's defaults)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="first run one plain torch copy of MIB MiB (reference kernel of "
                         "known traffic for counter runs)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="print the traffic summary of two rocprofv3 --pmc runs and exit")
    ap.add_argument("--summarize-trace", metavar="KERNEL_STATS_CSV",
                    help="print the summary of a rocprofv3 --kernel-trace --stats run and exit")
    ap.add_argument("--cmd", nargs="*", default=[], help="command line(s) quoted in a summary")
    args = ap.parse_args()
    if args.summarize_pmc:
        cmds = args.cmd + ["", ""]
        print(summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1],
                            args.copy_calibration or 1024, cmds[0], cmds[1], args.workload))
        return
    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace, (args.cmd + [""])[0], args.workload))
        return
    if args.gpus != 1:
        print("bench.py measures one GPU's share of the path; the multi-GPU collectives are "
              "not part of this build, so --gpus %d is not supported (use --gpus 1)"
              % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2609_20359_amd as P
    import synth.buffers as B
    from synth import workloads as W

    from paper_2609_20359_amd import runner

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    P.lib()
    if args.blocks_per_cu:
        P.set_blocks_per_cu(args.blocks_per_cu)
    w = W.ALL[args.workload]()
    log("workload", w.describe())
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    t0 = time.perf_counter()
    place_fn, placement = PLACEMENTS[args.placement]
    place = getattr(P, place_fn) if place_fn else None
    # the live probe places its streams the same way (stagger 0: one each)
    stagger = P.arena.STRIDE if args.placement == "staggered" else 0
    dev = B.DeviceInputs(w, place=place)
    torch.cuda.synchronize()
    log("inputs resident: %.1f GB in %.1f s (%s)" % (
        dev.bytes() / 1e9, time.perf_counter() - t0, placement))

    if args.copy_calibration:
        src = torch.empty(args.copy_calibration << 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        src.fill_(1.0)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log("copy calibration: %d MiB copied" % args.copy_calibration)
        del src, dst

    stream = torch.cuda.current_stream()
    K, Wm = args.steps, args.warmup
    # phase events only time the kernels between them: three per round (before
    # the first local step, before FedAvg, after it), recorded without the
    # system-scope cache fence, which would add a cache write-back per event
    events = [P.HipEvents(3, P.HIP_EVENT_DISABLE_SYSTEM_FENCE) for _ in range(K)]

    def phase_handles(ev):
        h = ev.handles
        return [h[0]] + [None] * (w.A - 1) + [h[1], h[2]]

    # every round also returns the per-segment sums of squares of each local
    # step's reduced gradient (A x n_seg floats)
    seg_sumsq = torch.empty(w.A * w.n_seg, dtype=torch.float32, device="cuda")
    for i in range(Wm):
        runner.gpu_round(lay, w, dev, seg_sumsq=seg_sumsq,
                         cfg=runner.round_cfg(w, w.step0 + w.A * i, dev=dev))
    torch.cuda.synchronize()
    log("warmup done (%d rounds)" % Wm)

    cfgs = [runner.round_cfg(w, w.step0 + w.A * (Wm + k), phase_events=phase_handles(events[k]),
                             dev=dev) for k in range(K)]
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    start.record(stream)
    for k in range(K):
        runner.gpu_round(lay, w, dev, seg_sumsq=seg_sumsq, cfg=cfgs[k])
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    total_ms = start.elapsed_time(stop)
    ms_round = total_ms / K
    round_ms = sorted(events[k].elapsed_ms(0, 2) for k in range(K))
    mid = K // 2
    median_ms = round_ms[mid] if K % 2 else 0.5 * (round_ms[mid - 1] + round_ms[mid])
    # the A local steps of a round lie between its first two events
    steps_ms = [events[k].elapsed_ms(0, 1) for k in range(K)]
    fed_ms = [events[k].elapsed_ms(1, 2) for k in range(K)]
    avg_step = sum(steps_ms) / (len(steps_ms) * w.A)
    avg_fed = sum(fed_ms) / len(fed_ms)
    log("timed %d rounds: %.3f ms/round (wall %.3f s); local step %.3f ms, fedavg %.3f ms"
        % (K, ms_round, wall, avg_step, avg_fed))

    bytes_round = w.round_bytes()
    gbs = bytes_round / (ms_round * 1e-3) / 1e9
    step_bytes = w.n * w.step_bytes_per_param()
    fed_bytes = w.n * w.fedavg_bytes_per_param()
    achieved = step_bytes / (avg_step * 1e-3) / 1e9
    src_hash = kernel_source_hash()
    traffic = read_traffic(args.workload, src_hash)
    out = {
        "metric": METRIC,
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": Wm,
        "ms_per_step": round(ms_round, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": dict(workload=w.name, n_params=w.n, segments=w.n_seg, R=w.R, G=w.G, A=w.A,
                       storage="bf16 gradients/replicas/working copy, fp32 master/m/v",
                       placement=placement,
                       bytes_per_round=bytes_round, parallelism="one GPU's shard"),
        "pct_of_peak": round(100.0 * gbs / PEAK_HBM_GBS, 2),
        "params_per_s": round(w.n / (ms_round * 1e-3), 1),
        "phases_ms": dict(local_step=round(avg_step, 4), fedavg=round(avg_fed, 4),
                          fedavg_gbs=round(fed_bytes / (avg_fed * 1e-3) / 1e9, 2)),
        "round_ms": dict(median=round(median_ms, 4),
                         min=round(round_ms[0], 4), max=round(round_ms[-1], 4)),
        "roofline": {
            "bound": "hbm",
            "kernel": step_label(w),
            "achieved": round(achieved, 2),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4),
            "traffic": traffic,
            "algorithmic_bytes": step_bytes,
            "kernel_source_hash": src_hash,
            "probe_reference": probe_reference(w, achieved),
        },
    }
    del dev
    torch.cuda.empty_cache()
    if not args.no_probe:
        out["roofline"]["probe_live"] = probe_live(w, achieved, stagger)
        if out["roofline"]["probe_live"]:
            log("live probe: %s at %.1f GB/s on this box" % (
                out["roofline"]["probe_live"]["pattern"], out["roofline"]["probe_live"]["gbs"]))
    if not args.no_cpu:
        log("cpu baseline: oracle on %d elements" % args.cpu_sample)
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_sample, args.cpu_seconds)
        log("cpu baseline done: %d rounds in %.1f s" % (out["cpu_baseline"]["rounds"],
                                                        out["cpu_baseline"]["seconds"]))
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)
    for e in events:
        e.close()
    lay.close()


if __name__ == "__main__":
    main()
