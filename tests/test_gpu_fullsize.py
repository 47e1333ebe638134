"""GPU parity at the workloads' full sizes, in the launch configuration and
the array placement the benchmark uses: one round on the whole shard, then
every element of the result compared with the oracle.

The oracle runs chunk by chunk (64 Mi elements) on the host's threads.  Each
chunk's inputs are the generator's values for that span: produced by the
generator's device build into a scratch tensor that the library never
touches, copied to the host, and spot-checked against the host build at
random indices of every array of every chunk (the two builds evaluate one
source; test_gpu_parity.test_generator_device_matches_host compares them
element by element).  Expected values
come only from the oracle.  A clipped round's coefficient depends on the
whole shard, so the oracle first streams each step's whole-shard sum of
squares the same way.

Every test writes one progress line per chunk to gpurun_out/ so that a long
comparison is visibly alive."""
import os
import time

import numpy as np
import pytest

import harness as H
import synth.buffers as B
from synth import workloads as W

pytestmark = pytest.mark.gpu

WORKLOADS = ["llama8b_s8", "fedavg_heavy", "hsdp_s4", "stress", "hsdp_s4_h2", "hsdp_s4_h2_recv",
             "llama8b_s8_outer", "llama8b_s8_clip"]
CHUNK = 1 << 26
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _say(*a):
    msg = " ".join(str(x) for x in a)
    print("[gpu-fullsize]", msg, flush=True)
    try:
        os.makedirs(os.path.join(ROOT, "gpurun_out"), exist_ok=True)
        with open(os.path.join(ROOT, "gpurun_out", "progress_fullsize.log"), "a") as f:
            f.write("%s %s\n" % (time.strftime("%H:%M:%S"), msg))
    except OSError:
        pass


@pytest.fixture(scope="module")
def env():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import oracle
    import paper_2609_20359_amd as P

    P.lib()
    return dict(torch=torch, P=P, orc=oracle.Oracle())


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", WORKLOADS)
def test_full_size_round_whole_shard(env, name):
    _whole_shard(env, W.ALL[name](), name)


@pytest.mark.timeout(900)
def test_beyond_int32_element_indices(env):
    """2^31 + 2053 elements: indices past the int32 range, a segment boundary
    3 elements past 2^31 (inside a tile), a 5-element ragged tail, and a
    short segment that straddles 2^31 itself."""
    n = (1 << 31) + 2053
    cuts = [0, 1 << 30, (1 << 31) - 700, (1 << 31) + 3, n]
    w = W.make_workload("beyond_int32", np.diff(cuts), [1, 0, 1, 1], R=2, G=2, A=1, step0=3,
                        weights=np.array([1.0, 3.0], np.float32))
    _whole_shard(env, w, "beyond_int32")


def _whole_shard(env, w, name):
    torch, P, orc = env["torch"], env["P"], env["orc"]
    _say(name, w.describe())
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    dev = B.DeviceInputs(w, place=P.place_arrays)      # the benchmark's placement
    ss = torch.full((w.A * w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
    H.gpu_round(P, lay, w, dev, seg_sumsq=ss)
    torch.cuda.synchronize()
    _say(name, "gpu round done")
    ss_gpu = ss.cpu().numpy()
    assert bool((ss >= 0).all()), "negative or unwritten per-segment sum of squares"
    lay.close()

    # keep only the results; the inputs are regenerated per chunk
    keep = dict(master=dev.master, m=dev.m, v=dev.v, working=dev.working)
    if w.outer is not None:
        keep.update(prev=dev.prev, buf=dev.buf)
    del dev
    torch.cuda.empty_cache()

    def state(k, lo, hi):
        t = keep[k][lo:hi]
        return H.to_u16(t) if k == "working" else t.cpu().numpy()

    filler = B.DeviceSpanFiller(min(CHUNK, w.n))
    totals = None
    if w.max_grad_norm > 0:
        totals = H.clip_totals(orc, w, chunk=CHUNK, say=lambda m: _say(name, m),
                               fill=lambda sp, lo, k: filler.fill(sp, lo, lo + k))
        _say(name, "clip coefficients", [orc.clip_coef(t, w.max_grad_norm) for t in totals[:1]])
    t0 = time.time()
    worst = H.whole_shard_parity(orc, w, state, ss_gpu, lambda lo, hi: filler.host_inputs(w, lo, hi),
                                 chunk=CHUNK, clip_totals=totals, say=lambda m: _say(name, m))
    _say(name, "ok: all %d elements bitwise equal to the oracle (%.1f s; %d generator values "
         "spot-checked against the host build); largest errors %s"
         % (w.n, time.time() - t0, filler.checked, worst))
