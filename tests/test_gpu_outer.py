"""GPU parity of the outer optimiser step (fl_fedopt, fl_round_outer)
against the oracle."""
import numpy as np
import pytest

import harness as H
import synth.buffers as B
from synth import workloads as W

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[gpu-outer]", *a, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import oracle
    import paper_2609_20359_amd as P

    P.lib()
    return dict(torch=torch, P=P, orc=oracle.Oracle())


def _workload(n, R, G, A, outer, seed):
    r = np.random.default_rng(seed)
    k = int(r.integers(1, min(n, 25) + 1))
    cuts = np.sort(r.choice(np.arange(1, n), size=k - 1, replace=False)) if k > 1 else []
    off = np.concatenate([[0], cuts, [n]]).astype(np.int64)
    flags = r.integers(0, 2, off.size - 1).astype(np.uint8)
    return W.make_workload("outer_n%d" % n, np.diff(off), flags, R=R, G=G, A=A,
                           weights=r.uniform(0.2, 3.0, G).astype(np.float32),
                           self_group=int(r.integers(0, G)), step0=int(r.integers(1, 40)),
                           outer=outer)


OUTERS = [dict(lr=0.7, momentum=0.9, nesterov=True), dict(lr=1.0, momentum=0.0, nesterov=True),
          dict(lr=0.4, momentum=0.6, nesterov=False)]


@pytest.mark.parametrize("n,R,G,A,oi", [
    (1, 1, 1, 1, 0), (2049, 3, 3, 2, 0), (100_003, 4, 4, 2, 1), (262_147, 8, 17, 1, 2),
    (7777, 2, 2, 3, 2),
])
def test_round_outer_two_rounds(env, n, R, G, A, oi):
    """Two rounds in a row (the outer state carries over) match the oracle
    bitwise."""
    torch, P, orc = env["torch"], env["P"], env["orc"]
    w = _workload(n, R, G, A, OUTERS[oi], seed=n + R + 5 * G)
    tag = "outer n=%d R=%d G=%d A=%d %s" % (n, R, G, A, OUTERS[oi])
    _say(tag)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    dev = B.DeviceInputs(w)
    host = B.HostInputs(w)
    for rnd in range(2):
        ss = torch.full((w.A * w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
        H.gpu_round(P, lay, w, dev, seg_sumsq=ss, cfg=H.round_cfg(P, w, w.step0 + rnd * w.A))
        w2 = W.Workload(**{**w.__dict__, "step0": w.step0 + rnd * w.A})
        ss_ref = H.oracle_round(orc, w2, host, want_sumsq=True)
        torch.cuda.synchronize()
        got = dict(master=dev.master.cpu().numpy(), m=dev.m.cpu().numpy(), v=dev.v.cpu().numpy(),
                   working=H.to_u16(dev.working))
        H.assert_state_parity(tag + " round %d" % rnd, got,
                              dict(master=host.master, m=host.m, v=host.v, working=host.working),
                              bitwise=True)
        H.assert_state_parity(tag + " outer state", dict(master=dev.prev.cpu().numpy(),
                                                         m=dev.buf.cpu().numpy()),
                              dict(master=host.prev, m=host.buf), bitwise=True)
        H.assert_sumsq(tag, ss.cpu().numpy(), ss_ref.reshape(-1))
    lay.close()


def test_fedopt_standalone_in_place(env):
    torch, P, orc = env["torch"], env["P"], env["orc"]
    w = _workload(150_001, 2, 4, 1, OUTERS[0], seed=1)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    dev = B.DeviceInputs(w)
    host = B.HostInputs(w)
    dev.buf.copy_(torch.from_numpy((np.random.default_rng(2).standard_normal(w.n) * 1e-4)
                                   .astype(np.float32)))
    host.buf[:] = dev.buf.cpu().numpy()
    reps_dev = [dev.working if x is None else x for x in dev.replicas]
    reps_host = [host.working if x is None else x for x in host.replicas]
    mref, wref = orc.fedopt(reps_host, w.weights, w.outer, host.prev, host.buf)
    P.fl_fedopt(lay, reps_dev, w.weights, w.outer, dev.prev, dev.buf, dev.master, dev.working,
                replica_fp=[lay.fingerprint] * w.G)
    torch.cuda.synchronize()
    for got, ref in ((dev.master, mref), (dev.prev, host.prev), (dev.buf, host.buf)):
        assert np.array_equal(got.cpu().numpy().view(np.uint32), ref.view(np.uint32))
    assert np.array_equal(H.to_u16(dev.working), wref)
    lay.close()


def test_round_outer_equals_chain(env):
    torch, P = env["torch"], env["P"]
    w = _workload(200_003, 4, 3, 2, OUTERS[0], seed=3)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    a, b = B.DeviceInputs(w), B.DeviceInputs(w)
    H.gpu_round(P, lay, w, a)
    for s in range(w.A):
        P.fl_local_step(lay, w.hp, w.step0 + s, b.grads[s * w.R:(s + 1) * w.R], w.grad_scale,
                        b.master, b.m, b.v, b.working)
    reps = [b.working if k == w.self_group else b.replicas[k] for k in range(w.G)]
    P.fl_fedopt(lay, reps, w.weights, w.outer, b.prev, b.buf, b.master, b.working)
    torch.cuda.synchronize()
    for k in ("master", "m", "v", "working", "prev", "buf"):
        assert torch.equal(getattr(a, k).view(torch.int16), getattr(b, k).view(torch.int16)), k
    lay.close()


def test_outer_errors(env):
    torch, P = env["torch"], env["P"]
    w = _workload(5000, 2, 2, 1, OUTERS[0], seed=4)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    d = B.DeviceInputs(w)
    cfg = H.round_cfg(P, w)

    def status(fn):
        try:
            fn()
        except P.FlError as e:
            return e.status
        return 0

    run = lambda o, prev=d.prev, buf=d.buf: P.fl_round_outer(  # noqa: E731
        lay, cfg, o, d.grads, d.replicas, prev, buf, d.master, d.m, d.v, d.working)
    assert status(lambda: run(dict(lr=0.7, momentum=1.5, nesterov=True))) == -1
    assert status(lambda: run(dict(lr=-1.0, momentum=0.5, nesterov=True))) == -1
    assert status(lambda: run(dict(lr=float("nan"), momentum=0.5, nesterov=True))) == -1
    assert status(lambda: run(OUTERS[0], prev=d.buf)) == -1
    assert status(lambda: run(OUTERS[0], prev=d.master)) == -1
    assert status(lambda: run(OUTERS[0], buf=None)) == -1
    torch.cuda.synchronize()
    lay.close()
