"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark uses: one fl_round on the whole shard, then the oracle on sampled
elements (every segment's first and last two elements, the tail, all of a few
short segments, and uniform random draws), plus properties that hold at any
size.  Sampled inputs are regenerated on the host by the same counter-based
generator; expected values come only from the oracle.  A clipped workload's
coefficient depends on the whole shard, so the oracle first streams each
step's whole-shard sum of squares over host-regenerated chunks."""
import numpy as np
import pytest

import harness as H
import synth.buffers as B
from synth import workloads as W

pytestmark = pytest.mark.gpu

WORKLOADS = ["llama8b_s8", "fedavg_heavy", "hsdp_s4", "stress", "hsdp_s4_h2", "hsdp_s4_h2_recv",
             "llama8b_s8_outer", "llama8b_s8_clip"]


def _say(*a):
    print("[gpu-fullsize]", *a, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import oracle
    import paper_2609_20359_amd as P

    P.lib()
    return dict(torch=torch, P=P, orc=oracle.Oracle())


@pytest.mark.parametrize("name", WORKLOADS)
def test_full_size_round_sampled(env, name):
    _sampled_parity(env, W.ALL[name](), name)


def test_beyond_int32_element_indices(env):
    """2^31 + 2053 elements: indices past the int32 range, a segment boundary
    3 elements past 2^31 (inside a tile), a 5-element ragged tail, and a
    short segment that straddles 2^31 itself."""
    n = (1 << 31) + 2053
    cuts = [0, 1 << 30, (1 << 31) - 700, (1 << 31) + 3, n]
    w = W.make_workload("beyond_int32", np.diff(cuts), [1, 0, 1, 1], R=2, G=2, A=1, step0=3,
                        weights=np.array([1.0, 3.0], np.float32))
    _sampled_parity(env, w, "beyond_int32")


def _sampled_parity(env, w, name):
    torch, P, orc = env["torch"], env["P"], env["orc"]
    _say(name, w.describe())
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    dev = B.DeviceInputs(w)
    ss = torch.full((w.A * w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
    H.gpu_round(P, lay, w, dev, seg_sumsq=ss)
    torch.cuda.synchronize()
    _say(name, "gpu round done")

    # properties at full size
    assert torch.equal(dev.master.to(torch.bfloat16).view(torch.int16),
                       dev.working.view(torch.int16)), "working != bf16(master)"
    for t in (dev.master, dev.m, dev.v):
        assert bool(torch.isfinite(t).all()), "non-finite state"
    assert bool((dev.v >= 0).all()), "negative second moment"
    assert bool((ss >= 0).all()), "negative or unwritten per-segment sum of squares"

    idx, full = W.sample_indices(w, n_random=1 << 16)
    idx_dev = torch.from_numpy(idx).cuda()
    got = dict(master=H.gather_f32(dev.master, idx_dev), m=H.gather_f32(dev.m, idx_dev),
               v=H.gather_f32(dev.v, idx_dev), working=H.gather_u16(dev.working, idx_dev))
    if w.outer is not None:
        got_outer = dict(master=H.gather_f32(dev.prev, idx_dev), m=H.gather_f32(dev.buf, idx_dev))
    ss_gpu = ss.cpu().numpy().reshape(w.A, w.n_seg)
    del dev
    torch.cuda.empty_cache()

    totals = H.clip_totals(orc, w, say=lambda m: _say(name, m)) if w.max_grad_norm > 0 else None
    if totals is not None:
        _say(name, "clip coefficients", [orc.clip_coef(t, w.max_grad_norm) for t in totals[:1]])
    host = B.HostInputs(w, idx)
    off, dec, cmap = H.compact_layout(w, idx, full)
    ss_ref = H.oracle_round(orc, w, host, seg_off=off, seg_decay=dec, want_sumsq=True,
                            clip_totals=totals)
    ref = dict(master=host.master, m=host.m, v=host.v, working=host.working)
    errs = H.assert_state_parity(name, got, ref, bitwise=True)
    if w.outer is not None:
        H.assert_state_parity(name + " outer state", got_outer,
                              dict(master=host.prev, m=host.buf), bitwise=True)
    for s, cs in cmap.items():
        H.assert_sumsq("%s seg %d" % (name, s), ss_gpu[:, s], ss_ref[:, cs])
    lay.close()
    _say(name, "ok: %d sampled elements, %d full segments, errors %s" % (idx.size, len(cmap), errs))
