"""GPU parity of global-norm gradient clipping (fl_grad_sumsq,
fl_local_step_clipped, fl_round_cfg.max_grad_norm) against the oracle."""
import numpy as np
import pytest

import harness as H
import synth.buffers as B
from synth import workloads as W

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[gpu-clip]", *a, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import oracle
    import paper_2609_20359_amd as P

    P.lib()
    return dict(torch=torch, P=P, orc=oracle.Oracle())


def _workload(n, R, A, max_norm, seed, **kw):
    r = np.random.default_rng(seed)
    k = int(r.integers(1, min(n, 25) + 1))
    cuts = np.sort(r.choice(np.arange(1, n), size=k - 1, replace=False)) if k > 1 else []
    off = np.concatenate([[0], cuts, [n]]).astype(np.int64)
    flags = r.integers(0, 2, off.size - 1).astype(np.uint8)
    return W.make_workload("clip_n%d" % n, np.diff(off), flags, R=R, G=2, A=A,
                           max_grad_norm=max_norm, step0=int(r.integers(1, 20)), **kw)


@pytest.mark.parametrize("n,R,A,max_norm,kind", [
    (1, 1, 1, 1e-5, "fsdp"), (2049, 3, 2, 1e-3, "fsdp"), (100_003, 4, 2, 0.05, "fsdp"),
    (100_003, 4, 2, 1e9, "fsdp"), (262_147, 8, 1, 0.02, "fsdp"), (50_001, 3, 2, 0.01, "hsdp"),
    (50_001, 3, 2, 0.01, "outer"), (1, 1, 2, 1e-5, "scratch"), (262_147, 8, 2, 0.02, "scratch"),
    (70_001, 16, 1, 1e9, "scratch"), (50_001, 6, 2, 0.01, "outer-scratch"),
])
def test_clipped_round_parity(env, n, R, A, max_norm, kind):
    torch, P, orc = env["torch"], env["P"], env["orc"]
    kw = {}
    if kind == "hsdp":
        kw = dict(H=3, replica=1, hsdp_member=True)
    if kind.startswith("outer"):
        kw = dict(outer=dict(lr=0.7, momentum=0.9, nesterov=True))
    if kind.endswith("scratch"):
        kw["clip_scratch"] = True
    w = _workload(n, R, A, max_norm, seed=n + R, **kw)
    tag = "clip %s n=%d R=%d A=%d max=%g" % (kind, n, R, A, max_norm)
    _say(tag)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    dev = B.DeviceInputs(w)
    ss = torch.full((w.A * w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
    H.gpu_round(P, lay, w, dev, seg_sumsq=ss)
    torch.cuda.synchronize()
    host = B.HostInputs(w)
    ss_ref = H.oracle_round(orc, w, host, want_sumsq=True)
    H.assert_state_parity(tag, dict(master=dev.master.cpu().numpy(), m=dev.m.cpu().numpy(),
                                    v=dev.v.cpu().numpy(), working=H.to_u16(dev.working)),
                          dict(master=host.master, m=host.m, v=host.v, working=host.working),
                          bitwise=True)
    worst = H.assert_sumsq(tag, ss.cpu().numpy(), ss_ref.reshape(-1))
    _say(tag, "seg_sumsq worst rel err %.3g" % worst)
    lay.close()


@pytest.mark.parametrize("bad", [0x7FC0, 0x7F80, 0xFF80])
def test_clipped_round_with_a_nonfinite_gradient(env, bad):
    """One NaN or infinite bf16 value in the first step's first peer
    gradient: a NaN norm makes every clipped gradient NaN; an infinite norm
    gives a zero coefficient (NaN at the infinite entry itself), as
    clip_grad_norm_ does.  Compared with the oracle element by element (NaN
    positions, all other bits)."""
    torch, P, orc = env["torch"], env["P"], env["orc"]
    w = _workload(5003, 2, 2, 0.01, seed=13)
    tag = "clip nonfinite 0x%04X" % bad
    _say(tag)
    k = 1234
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    dev = B.DeviceInputs(w)
    dev.grad_arrays[w.grad_index[0]].view(torch.int16)[k] = bad - 0x10000 if bad > 0x7FFF else bad
    ss = torch.full((w.A * w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
    H.gpu_round(P, lay, w, dev, seg_sumsq=ss)
    torch.cuda.synchronize()
    host = B.HostInputs(w)
    host.grad_arrays[w.grad_index[0]][k] = bad
    ss_ref = H.oracle_round(orc, w, host, want_sumsq=True)
    got = dict(master=dev.master.cpu().numpy(), m=dev.m.cpu().numpy(), v=dev.v.cpu().numpy(),
               working=H.to_u16(dev.working))
    H.assert_state_parity(tag, got, dict(master=host.master, m=host.m, v=host.v,
                                         working=host.working), bitwise=True)
    H.assert_sumsq(tag, ss.cpu().numpy(), ss_ref.reshape(-1))
    n_nan = int(np.isnan(got["master"]).sum())
    assert n_nan == (w.n if bad == 0x7FC0 else 1), "%s: %d NaNs in master" % (tag, n_nan)
    lay.close()


@pytest.mark.parametrize("R", [1, 3, 8, 16])
def test_scratch_path_is_bitwise_the_two_read_path(env, R):
    """With a gradient scratch the round reads the peer gradients once and
    takes the AdamW-only pass; state and per-segment sums equal the round
    without it bit for bit."""
    torch, P = env["torch"], env["P"]
    w = _workload(200_011, R, 3, 0.03, seed=20 + R)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    a, b = B.DeviceInputs(w), B.DeviceInputs(w)
    scratch = torch.empty(w.n, dtype=torch.float32, device="cuda")
    ssa = torch.empty(w.A * w.n_seg, dtype=torch.float32, device="cuda")
    ssb = torch.empty_like(ssa)
    H.gpu_round(P, lay, w, a, seg_sumsq=ssa)
    cfg = P.make_round_cfg(w.R, w.G, w.A, w.weights, w.hp, self_group=w.self_group,
                           grad_scale=w.grad_scale, step0=w.step0,
                           max_grad_norm=w.max_grad_norm, grad_scratch=scratch)
    P.fl_round(lay, cfg, b.grads, b.replicas, b.master, b.m, b.v, b.working, seg_sumsq=ssb)
    torch.cuda.synchronize()
    for k in ("master", "m", "v", "working"):
        assert torch.equal(getattr(a, k).view(torch.int16), getattr(b, k).view(torch.int16)), k
    assert torch.equal(ssa.view(torch.int32), ssb.view(torch.int32)), "per-segment sums"
    bad = P.make_round_cfg(w.R, w.G, w.A, w.weights, w.hp, max_grad_norm=w.max_grad_norm,
                           grad_scratch=b.m)
    with pytest.raises(P.FlError) as e:
        P.fl_round(lay, bad, b.grads, b.replicas, b.master, b.m, b.v, b.working)
    assert e.value.status == -1
    short = P.make_round_cfg(w.R, w.G, w.A, w.weights, w.hp, max_grad_norm=w.max_grad_norm,
                             grad_scratch=scratch[:-8])
    with pytest.raises(ValueError):
        P.fl_round(lay, short, b.grads, b.replicas, b.master, b.m, b.v, b.working)
    lay.close()


def test_grad_sumsq_then_clipped_step_equals_round(env):
    """The two-call form (sum of squares, then the clipped step: what a
    multi-GPU caller does around its all-reduce) is bitwise fl_round's."""
    torch, P, orc = env["torch"], env["P"], env["orc"]
    w = _workload(300_007, 4, 2, 0.05, seed=11)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    a, b = B.DeviceInputs(w), B.DeviceInputs(w)
    H.gpu_round(P, lay, w, a)
    total = torch.empty(1, dtype=torch.float64, device="cuda")
    seg = torch.empty(w.n_seg, dtype=torch.float32, device="cuda")
    host = B.HostInputs(w)
    for s in range(w.A):
        peers = b.grads[s * w.R:(s + 1) * w.R]
        P.fl_grad_sumsq(lay, peers, w.grad_scale, total, seg_sumsq=seg)
        torch.cuda.synchronize()
        g = orc.shard_reduce(host.grads[s * w.R:(s + 1) * w.R], w.grad_scale)
        want = orc.total_sumsq(g)
        assert abs(total.item() - want) <= 1e-12 * want, "whole-shard sum of squares"
        H.assert_sumsq("seg", seg.cpu().numpy(), orc.seg_sumsq(w.seg_offsets, g))
        P.fl_local_step_clipped(lay, w.hp, w.step0 + s, peers, w.grad_scale, total,
                                w.max_grad_norm, b.master, b.m, b.v, b.working)
    reps = [b.working if k == w.self_group else b.replicas[k] for k in range(w.G)]
    P.fl_fedavg(lay, reps, w.weights, b.master, b.working)
    torch.cuda.synchronize()
    for k in ("master", "m", "v", "working"):
        assert torch.equal(getattr(a, k).view(torch.int16), getattr(b, k).view(torch.int16)), k
    lay.close()


def test_clip_errors(env):
    torch, P = env["torch"], env["P"]
    w = _workload(5000, 2, 1, 0.1, seed=12)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    d = B.DeviceInputs(w)
    total = torch.zeros(1, dtype=torch.float64, device="cuda")

    def status(fn):
        try:
            fn()
        except P.FlError as e:
            return e.status
        return 0

    step = lambda mx, tot=total: P.fl_local_step_clipped(  # noqa: E731
        lay, w.hp, 1, d.grads[:2], 0.5, tot, mx, d.master, d.m, d.v, d.working)
    assert status(lambda: step(0.0)) == -1
    assert status(lambda: step(float("inf"))) == -1
    assert status(lambda: step(1.0, tot=None)) == -1
    bad = P.make_round_cfg(w.R, w.G, w.A, w.weights, w.hp, max_grad_norm=float("nan"))
    assert status(lambda: H.gpu_round(P, lay, w, d, cfg=bad)) == -1
    assert status(lambda: P.fl_grad_sumsq(lay, d.grads[:2], 0.5, None)) == -1
    torch.cuda.synchronize()
    lay.close()
