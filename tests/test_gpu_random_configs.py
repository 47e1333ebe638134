"""GPU parity over seeded random configurations of the whole round: shard
length and segments, R, G, A, AdamW hyperparameters, weights, self group,
step0, FL+HSDP replicas (member or receiver), the outer step, clipping (with
and without the gradient scratch) and per-step learning rates, each drawn
independently.  Every case is compared with the oracle element by element:
master, m, v and working copy bitwise, the outer state bitwise, and the
per-segment sums of squares within their tolerance."""
import numpy as np
import pytest

import harness as H
import synth.buffers as B
from synth import workloads as W

pytestmark = pytest.mark.gpu

N_CASES = 128


def _say(*a):
    print("[gpu-random]", *a, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import oracle
    import paper_2609_20359_amd as P

    P.lib()
    return dict(torch=torch, P=P, orc=oracle.Oracle())


def _case(k):
    r = np.random.default_rng(7000 + k)
    n = int(r.choice([1, 7, 2048, 2049, 6143, int(r.integers(1, 400_000))]))
    nseg = int(r.integers(1, min(n, 40) + 1))
    cuts = np.sort(r.choice(np.arange(1, n), size=nseg - 1, replace=False)) if nseg > 1 else []
    off = np.concatenate([[0], cuts, [n]]).astype(np.int64)
    flags = r.integers(0, 2, off.size - 1).astype(np.uint8)
    R = int(r.choice([1, 2, 3, 4, 5, 8, 13, 16, 20]))
    G = int(r.integers(1, 10))
    A = int(r.integers(1, 4))
    Hh = int(r.choice([1, 1, 2, 3]))
    outer = None
    if Hh == 1 and r.random() < 0.4:
        outer = dict(lr=float(r.uniform(0.3, 1.0)), momentum=float(r.uniform(0.0, 0.95)),
                     nesterov=bool(r.random() < 0.5))
    clip = 0.0 if r.random() < 0.5 else float(10 ** r.uniform(-4, 0))
    hp = dict(lr=float(10 ** r.uniform(-5, -2)), beta1=float(r.uniform(0.0, 0.99)),
              beta2=float(r.uniform(0.9, 0.9999)), eps=float(10 ** r.uniform(-8, -3)),
              weight_decay=float(r.uniform(0.0, 0.2)))
    step_lr = None if r.random() < 0.5 else [float(x) for x in
                                             r.uniform(0.0, 1e-3, A).astype(np.float32)]
    w = W.make_workload("random_%d" % k, np.diff(off), flags, R=R, G=G, A=A,
                        weights=r.uniform(0.1, 5.0, G).astype(np.float32), seed=k,
                        distinct_grads=bool(r.random() < 0.5), student=bool(r.random() < 0.3),
                        hp=hp, self_group=int(r.integers(0, G)), step0=int(r.integers(1, 100)),
                        H=Hh, replica=int(r.integers(0, Hh)),
                        hsdp_member=bool(Hh == 1 or r.random() < 0.7), outer=outer,
                        max_grad_norm=clip, clip_scratch=bool(clip > 0 and r.random() < 0.5))
    return w, step_lr


@pytest.mark.parametrize("k", range(N_CASES))
def test_random_round_configuration(env, k):
    torch, P, orc = env["torch"], env["P"], env["orc"]
    w, step_lr = _case(k)
    tag = "case %d %s step_lr=%s hp=%s" % (k, w.describe(), step_lr is not None, w.hp)
    _say(tag)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    dev = B.DeviceInputs(w)
    ss = torch.full((w.A * w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
    H.gpu_round(P, lay, w, dev, seg_sumsq=ss, cfg=H.round_cfg(P, w, dev=dev, step_lr=step_lr))
    torch.cuda.synchronize()
    host = B.HostInputs(w)
    ss_ref = H.oracle_round(orc, w, host, want_sumsq=True, step_lr=step_lr)
    got = dict(master=dev.master.cpu().numpy(), m=dev.m.cpu().numpy(), v=dev.v.cpu().numpy(),
               working=H.to_u16(dev.working))
    H.assert_state_parity(tag, got, dict(master=host.master, m=host.m, v=host.v,
                                         working=host.working), bitwise=True)
    if w.outer is not None:
        H.assert_state_parity(tag + " outer state", dict(master=dev.prev.cpu().numpy(),
                                                         m=dev.buf.cpu().numpy()),
                              dict(master=host.prev, m=host.buf), bitwise=True)
    H.assert_sumsq(tag, ss.cpu().numpy(), ss_ref.reshape(-1))
    lay.close()


def _large_case(k):
    r = np.random.default_rng(90000 + k)
    n = int(r.integers(2_000_000, 8_000_000))
    nseg = int(r.integers(1, 400))
    cuts = np.sort(r.choice(np.arange(1, n), size=nseg - 1, replace=False)) if nseg > 1 else []
    off = np.concatenate([[0], cuts, [n]]).astype(np.int64)
    flags = r.integers(0, 2, off.size - 1).astype(np.uint8)
    R = int(r.choice([1, 3, 4, 8, 12, 16]))
    G = int(r.integers(1, 8))
    Hh = (1, 2, 1, 3)[k % 4]                    # FL+FSDP and FL+HSDP cases
    outer = None if Hh > 1 or r.random() < 0.5 else W.DILOCO_OUTER
    clip = 0.0 if r.random() < 0.5 else float(10 ** r.uniform(-3, 0))
    return W.make_workload("large_%d" % k, np.diff(off), flags, R=R, G=G, A=int(r.integers(1, 3)),
                           seed=k, weights=r.uniform(0.1, 5.0, G).astype(np.float32),
                           self_group=int(r.integers(0, G)), step0=int(r.integers(1, 500)), H=Hh,
                           replica=int(r.integers(0, Hh)),
                           hsdp_member=bool(Hh == 1 or k % 4 == 1), outer=outer,
                           max_grad_norm=clip, clip_scratch=bool(clip > 0 and r.random() < 0.5))


@pytest.mark.parametrize("k", range(4))
def test_random_large_configuration(env, k):
    """Random configurations of 2-8 million elements and up to 400 segments,
    compared with the oracle on the whole shard."""
    torch, P, orc = env["torch"], env["P"], env["orc"]
    w = _large_case(k)
    tag = "large case %d %s" % (k, w.describe())
    _say(tag)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    dev = B.DeviceInputs(w)
    ss = torch.full((w.A * w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
    H.gpu_round(P, lay, w, dev, seg_sumsq=ss)
    torch.cuda.synchronize()
    host = B.HostInputs(w)
    ss_ref = H.oracle_round(orc, w, host, want_sumsq=True)
    got = dict(master=dev.master.cpu().numpy(), m=dev.m.cpu().numpy(), v=dev.v.cpu().numpy(),
               working=H.to_u16(dev.working))
    H.assert_state_parity(tag, got, dict(master=host.master, m=host.m, v=host.v,
                                         working=host.working), bitwise=True)
    if w.outer is not None:
        H.assert_state_parity(tag + " outer state", dict(master=dev.prev.cpu().numpy(),
                                                         m=dev.buf.cpu().numpy()),
                              dict(master=host.prev, m=host.buf), bitwise=True)
    H.assert_sumsq(tag, ss.cpu().numpy(), ss_ref.reshape(-1))
    lay.close()
