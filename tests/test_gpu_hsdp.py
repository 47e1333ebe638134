"""GPU parity of the FL+HSDP entry points (two-tier gradient average, wire
reduction, broadcast receive, whole FL+HSDP rounds) against the oracle."""
import numpy as np
import pytest

import harness as H
import synth.buffers as B
from synth import workloads as W

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[gpu-hsdp]", *a, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import oracle
    import paper_2609_20359_amd as P

    P.lib()
    return dict(torch=torch, P=P, orc=oracle.Oracle())


def _state(dev):
    return dict(master=dev.master.cpu().numpy(), m=dev.m.cpu().numpy(), v=dev.v.cpu().numpy(),
                working=H.to_u16(dev.working))


def _workload(n, R, Hh, A, member, seed):
    r = np.random.default_rng(seed)
    k = int(r.integers(1, min(n, 30) + 1))
    cuts = np.sort(r.choice(np.arange(1, n), size=k - 1, replace=False)) if k > 1 else []
    off = np.concatenate([[0], cuts, [n]]).astype(np.int64)
    flags = r.integers(0, 2, off.size - 1).astype(np.uint8)
    return W.make_workload("hsdp_n%d_r%d_h%d" % (n, R, Hh), np.diff(off), flags, R=R, G=3, A=A,
                           weights=r.integers(1, 9, 3).astype(np.float32), H=Hh,
                           replica=int(r.integers(0, Hh)), hsdp_member=bool(member),
                           self_group=int(r.integers(0, 3)), step0=int(r.integers(1, 30)))


@pytest.mark.parametrize("n,R,Hh,A,member", [
    (1, 1, 2, 1, 1), (2049, 3, 2, 2, 1), (2049, 3, 2, 2, 0), (100_003, 4, 3, 2, 0),
    (262_147, 8, 4, 1, 1), (6143, 2, 1, 2, 1), (50_000, 5, 17, 1, 1),
])
def test_round_hsdp_parity(env, n, R, Hh, A, member):
    torch, P, orc = env["torch"], env["P"], env["orc"]
    w = _workload(n, R, Hh, A, member, seed=n + 7 * R + Hh)
    tag = "hsdp n=%d R=%d H=%d A=%d member=%d" % (n, R, Hh, A, member)
    _say(tag)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    dev = B.DeviceInputs(w)
    ss = torch.full((w.A * w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
    H.gpu_round(P, lay, w, dev, seg_sumsq=ss)
    torch.cuda.synchronize()
    host = B.HostInputs(w)
    ss_ref = H.oracle_round(orc, w, host, want_sumsq=True)
    H.assert_state_parity(tag, _state(dev), dict(master=host.master, m=host.m, v=host.v,
                                                 working=host.working), bitwise=True)
    H.assert_sumsq(tag, ss.cpu().numpy(), ss_ref.reshape(-1))
    lay.close()


def test_one_replica_is_fl_fsdp(env):
    torch, P = env["torch"], env["P"]
    w = _workload(70_001, 4, 1, 3, 1, seed=3)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    a, b = B.DeviceInputs(w), B.DeviceInputs(w)
    cfg = H.round_cfg(P, w)
    P.fl_round_hsdp(lay, cfg, P.make_hsdp_cfg(1, 0, 1.0, True), a.grads, None, None, a.replicas,
                    None, a.master, a.m, a.v, a.working)
    P.fl_round(lay, cfg, b.grads, b.replicas, b.master, b.m, b.v, b.working)
    torch.cuda.synchronize()
    for k in ("master", "m", "v", "working"):
        assert torch.equal(getattr(a, k).view(torch.int16), getattr(b, k).view(torch.int16)), k
    lay.close()


def test_one_replica_clipped_with_scratch_is_fl_fsdp(env):
    """With one replica, a clipped FL+HSDP round with the gradient scratch is
    bitwise the clipped fl_round with the scratch."""
    torch, P = env["torch"], env["P"]
    w = _workload(70_001, 8, 1, 2, 1, seed=7)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    a, b = B.DeviceInputs(w), B.DeviceInputs(w)
    sa = torch.empty(w.n, dtype=torch.float32, device="cuda")
    sb = torch.empty_like(sa)
    mk = lambda s: P.make_round_cfg(w.R, w.G, w.A, w.weights, w.hp,  # noqa: E731
                                    self_group=w.self_group, grad_scale=w.grad_scale,
                                    step0=w.step0, max_grad_norm=0.01, grad_scratch=s)
    P.fl_round_hsdp(lay, mk(sa), P.make_hsdp_cfg(1, 0, 1.0, True), a.grads, None, None,
                    a.replicas, None, a.master, a.m, a.v, a.working)
    P.fl_round(lay, mk(sb), b.grads, b.replicas, b.master, b.m, b.v, b.working)
    torch.cuda.synchronize()
    for k in ("master", "m", "v", "working"):
        assert torch.equal(getattr(a, k).view(torch.int16), getattr(b, k).view(torch.int16)), k
    assert torch.equal(sa.view(torch.int32), sb.view(torch.int32)), "scratch not used alike"
    lay.close()


def test_wire_reduce_and_broadcast_receive(env):
    torch, P, orc = env["torch"], env["P"], env["orc"]
    w = _workload(123_457, 6, 2, 1, 0, seed=4)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    dev = B.DeviceInputs(w)
    host = B.HostInputs(w)
    wire = torch.empty(w.n, dtype=torch.bfloat16, device="cuda")
    P.fl_shard_reduce_wire(lay, dev.grads[:w.R], w.grad_scale, wire)
    P.fl_broadcast_recv(lay, dev.bcast, dev.master, dev.working)
    torch.cuda.synchronize()
    assert np.array_equal(H.to_u16(wire), orc.shard_reduce_wire(host.grads[:w.R], w.grad_scale))
    mref = np.zeros(w.n, np.float32)
    wref = np.zeros(w.n, np.uint16)
    orc.broadcast_recv(host.bcast, mref, wref)
    assert np.array_equal(dev.master.cpu().numpy().view(np.uint32), mref.view(np.uint32))
    assert np.array_equal(H.to_u16(dev.working), wref)
    lay.close()


def test_round_hsdp_equals_chain(env):
    """fl_round_hsdp is bitwise the chain of its parts."""
    torch, P = env["torch"], env["P"]
    w = _workload(300_001, 4, 3, 2, 1, seed=5)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    a, b = B.DeviceInputs(w), B.DeviceInputs(w)
    H.gpu_round(P, lay, w, a)
    for s in range(w.A):
        P.fl_shard_reduce_wire(lay, b.grads[s * w.R:(s + 1) * w.R], w.grad_scale, b.wire)
        wires = [b.wire if k == w.replica else b.replica_wires[s * w.H + k] for k in range(w.H)]
        P.fl_local_step(lay, w.hp, w.step0 + s, wires, 1.0 / w.H, b.master, b.m, b.v, b.working)
    reps = [b.working if k == w.self_group else b.replicas[k] for k in range(w.G)]
    P.fl_fedavg(lay, reps, w.weights, b.master, b.working)
    torch.cuda.synchronize()
    for k in ("master", "m", "v", "working"):
        assert torch.equal(getattr(a, k).view(torch.int16), getattr(b, k).view(torch.int16)), k
    lay.close()


def test_round_hsdp_errors(env):
    torch, P = env["torch"], env["P"]
    w = _workload(5000, 2, 2, 1, 1, seed=6)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    d = B.DeviceInputs(w)
    cfg = H.round_cfg(P, w)

    def status(hc, wires=d.replica_wires, wire=d.wire, reps=d.replicas, bcast=None):
        try:
            P.fl_round_hsdp(lay, cfg, hc, d.grads, wires, wire, reps, bcast, d.master, d.m, d.v,
                            d.working)
        except P.FlError as e:
            return e.status
        return 0

    assert status(P.make_hsdp_cfg(2, 2)) == -1            # replica out of range
    assert status(P.make_hsdp_cfg(65, 0)) == -1           # too many replicas
    assert status(P.make_hsdp_cfg(2, 0), wires=None) == -1
    assert status(P.make_hsdp_cfg(2, 0), wire=None) == -1
    assert status(P.make_hsdp_cfg(2, 0, fedavg_member=False)) == -1   # no broadcast buffer
    assert status(P.make_hsdp_cfg(2, 0), wire=d.working) == -1
    torch.cuda.synchronize()
    lay.close()
