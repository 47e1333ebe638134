"""fl_round_noalloc, the entry point for callers that cannot allocate: its
results equal fl_round's bit for bit, on two calls in a row (the second on a
smaller shard, with a different segment structure), it refuses a layout
whose workspace exceeds the static scratch before enqueueing anything, and a
round with per-segment sums captured into a HIP graph replays correctly."""
import numpy as np
import pytest

import harness as H
import synth.buffers as B
from synth import workloads as W

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[gpu-noalloc]", *a, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_20359_amd as P

    P.lib()
    return dict(torch=torch, P=P)


def _outputs(dev, ss):
    return dict(master=dev.master.cpu().numpy(), m=dev.m.cpu().numpy(), v=dev.v.cpu().numpy(),
                working=H.to_u16(dev.working), ss=ss.cpu().numpy())


def _bitwise(tag, a, b):
    for k in a:
        u = np.uint16 if k == "working" else np.uint32
        assert np.array_equal(np.asarray(a[k]).view(u), np.asarray(b[k]).view(u)), (tag, k)


def _round_pair(env, w):
    """The same round through fl_round_noalloc and through fl_round, each on
    its own copy of the inputs; returns both outputs."""
    torch, P = env["torch"], env["P"]
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    assert 0 < P.noalloc_workspace_bytes(lay) <= P.FL_NOALLOC_SCRATCH_BYTES
    d0, d1 = B.DeviceInputs(w), B.DeviceInputs(w)
    s0 = torch.full((w.A * w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
    s1 = torch.full((w.A * w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    cfg = H.round_cfg(P, w, dev=d0)
    P.fl_round_noalloc(lay, cfg, d0.grads, d0.replicas, d0.master, d0.m, d0.v, d0.working,
                       seg_sumsq=s0)
    cfg1 = H.round_cfg(P, w, dev=d1)
    P.fl_round(lay, cfg1, d1.grads, d1.replicas, d1.master, d1.m, d1.v, d1.working,
               seg_sumsq=s1)
    torch.cuda.synchronize()
    out = _outputs(d0, s0), _outputs(d1, s1)
    lay.close()
    return out


def test_noalloc_round_equals_fl_round_twice(env):
    # first call: 400k elements in 6 segments (each step's finalize carried by
    # the next kernel; per-segment sums); second: a smaller shard of 300
    # segments (separate finalize kernels) with clipping, in the same static
    # scratch
    w1 = W.make_workload("noalloc_a", [150000, 17, 2049, 100000, 3, 147931],
                         [1, 0, 1, 1, 0, 1], R=4, G=3, A=3, seed=3,
                         weights=np.array([1, 2, 1], np.float32))
    r = np.random.default_rng(41)
    sizes = r.integers(1, 400, 300)
    w2 = W.make_workload("noalloc_b", sizes, (np.arange(300) % 2).astype(np.uint8), R=3, G=2,
                         A=2, seed=4, max_grad_norm=1e-3)
    assert w2.n < w1.n
    for w in (w1, w2):
        _say(w.describe())
        a, b = _round_pair(env, w)
        _bitwise(w.name, a, b)
        assert np.all(a["ss"] >= 0)


def test_noalloc_refuses_an_oversized_workspace(env):
    """One-element segments make the workspace larger than the static
    scratch: FL_ERR_SCRATCH before anything runs (outputs untouched); the
    same call without per-segment sums or clipping needs no workspace and
    runs."""
    torch, P = env["torch"], env["P"]
    n = 1 << 20
    w = W.make_workload("noalloc_big", np.ones(n, np.int64), np.ones(n, np.uint8), R=2, G=2, A=1)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    assert P.noalloc_workspace_bytes(lay) > P.FL_NOALLOC_SCRATCH_BYTES
    d = B.DeviceInputs(w)
    ss = torch.full((w.A * w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
    before = d.master.clone()
    torch.cuda.synchronize()
    cfg = H.round_cfg(P, w)
    with pytest.raises(P.FlError) as e:
        P.fl_round_noalloc(lay, cfg, d.grads, d.replicas, d.master, d.m, d.v, d.working,
                           seg_sumsq=ss)
    assert e.value.status == -7
    torch.cuda.synchronize()
    assert torch.equal(before, d.master) and bool((ss == -1.0).all())
    P.fl_round_noalloc(lay, cfg, d.grads, d.replicas, d.master, d.m, d.v, d.working)
    torch.cuda.synchronize()
    assert not torch.equal(before, d.master)
    lay.close()


def test_noalloc_round_in_a_hip_graph(env):
    """fl_round_noalloc with per-segment sums captured once and replayed
    three times, with eager work and synchronisation between replays; every
    replay equals the eager fl_round of the same round."""
    torch, P = env["torch"], env["P"]
    w = W.make_workload("noalloc_graph", [60000, 33, 70001], [1, 0, 1], R=4, G=2, A=2, seed=8)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    eager, graphed = B.DeviceInputs(w), B.DeviceInputs(w)
    se = torch.zeros(w.A * w.n_seg, dtype=torch.float32, device="cuda")
    sg = torch.zeros(w.A * w.n_seg, dtype=torch.float32, device="cuda")
    cfg = H.round_cfg(P, w)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(g, stream=s):
        P.fl_round_noalloc(lay, cfg, graphed.grads, graphed.replicas, graphed.master, graphed.m,
                           graphed.v, graphed.working, seg_sumsq=sg)
    torch.cuda.synchronize()
    for rep in range(3):
        P.fl_round(lay, cfg, eager.grads, eager.replicas, eager.master, eager.m, eager.v,
                   eager.working, seg_sumsq=se)
        junk = torch.randn(1 << 20, device="cuda").sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        _bitwise("replay %d" % rep, _outputs(graphed, sg), _outputs(eager, se))
        del junk
    lay.close()
