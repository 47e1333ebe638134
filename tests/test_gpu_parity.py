"""GPU parity: the HIP path through the C ABI against the CPU oracle on the
same seeded inputs, element by element (sizes the oracle finishes quickly,
spanning many 2048-element tiles and ragged tails)."""
import numpy as np
import pytest

import harness as H
import synth
import synth.buffers  # noqa: F401
import synth.buffers as B
from synth import workloads as W

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[gpu-parity]", *a, flush=True)


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


def _host_state(host):
    return dict(master=host.master, m=host.m, v=host.v, working=host.working)


def _round_parity(env, w, tag, sumsq=True):
    torch, P, orc = env["torch"], env["P"], env["orc"]
    _say(tag, w.describe())
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    dev = synth.buffers.DeviceInputs(w)
    ss_dev = torch.full((w.A * max(w.n_seg, 1),), -1.0, dtype=torch.float32,
                        device="cuda") if sumsq else None
    H.gpu_round(P, lay, w, dev, seg_sumsq=ss_dev)
    torch.cuda.synchronize()
    host = synth.buffers.HostInputs(w)
    ss_ref = H.oracle_round(orc, w, host, want_sumsq=sumsq)
    errs = H.assert_state_parity(tag, _state(dev), _host_state(host), bitwise=True)
    if sumsq and w.n_seg:
        H.assert_sumsq(tag, ss_dev.cpu().numpy()[:w.A * w.n_seg], ss_ref.reshape(-1))
    lay.close()
    _say(tag, "ok", errs)


def test_generator_device_matches_host(env):
    torch = env["torch"]
    specs = [synth.spec(synth.NORMAL_F32, 1, 0, 0.0, 0.02),
             synth.spec(synth.NORMAL_BF16, 1000, 0, 0.0, 1e-3),
             synth.spec(synth.DRIFT_F32, 1, 0, 0.0, 0.02, stream2=2000, std2=1e-4),
             synth.spec(synth.DRIFT_BF16, 1, 3, 0.0, 0.02, stream2=2005, std2=1e-4),
             synth.spec(synth.STUDENT3_BF16, 1007, 0, 0.0, 1e-3, p_zero=0.05)]
    for sp in specs:
        for i0, n in ((0, 100_003), (987_654_321, 4097)):
            t = torch.empty(n, dtype=torch.bfloat16 if sp.is_bf16 else torch.float32,
                            device="cuda")
            synth.dev_fill(t, sp, i0)
            got = H.to_u16(t) if sp.is_bf16 else t.cpu().numpy().view(np.uint32)
            want = synth.host_fill(sp, i0, n)
            want = want if sp.is_bf16 else want.view(np.uint32)
            assert np.array_equal(got, want), "device generator differs from host for %r" % sp


def test_round_tiny_workload(env):
    _round_parity(env, W.tiny(), "tiny")


def test_round_stress_shaped_small(env):
    """The stress workload's structure (odd segment sizes, Student-t gradients
    with exact zeros, R = G = 16) at a size the oracle runs in seconds."""
    r = np.random.default_rng(5)
    sizes = r.integers(1, 4096, 300)
    sizes[sizes % 256 == 0] += 1
    flags = r.integers(0, 2, sizes.size).astype(np.uint8)
    u = r.uniform(0, 1, 16)
    w = W.make_workload("stress_small", sizes, flags, R=16, G=16, A=2,
                        weights=(u / u.sum()).astype(np.float32), student=True)
    _round_parity(env, w, "stress_small")


@pytest.mark.parametrize("n,R,G,A", [
    (1, 1, 1, 1), (7, 3, 2, 1), (8, 2, 3, 2), (9, 5, 1, 1), (2047, 4, 4, 1), (2048, 8, 8, 1),
    (2049, 16, 16, 1), (6143, 17, 17, 2), (100_003, 6, 5, 3), (262_147, 64, 64, 1),
    (5003, 2, 2, 32),
])
def test_round_ragged_shapes(env, n, R, G, A):
    r = np.random.default_rng(n + 31 * R + 7 * G)
    k = int(r.integers(1, min(n, 40) + 1))
    cuts = np.sort(r.choice(np.arange(1, n), size=k - 1, replace=False)) if k > 1 else []
    off = np.concatenate([[0], cuts, [n]]).astype(np.int64)
    sizes = np.diff(off)
    flags = r.integers(0, 2, sizes.size).astype(np.uint8)
    weights = r.integers(1, 17, G).astype(np.float32)
    w = W.make_workload("ragged_n%d" % n, sizes, flags, R=R, G=G, A=A, weights=weights,
                        self_group=int(r.integers(0, G)), step0=int(r.integers(1, 50)))
    _round_parity(env, w, "ragged n=%d R=%d G=%d A=%d" % (n, R, G, A))


def test_standalone_entry_points(env):
    """fl_shard_reduce, fl_adamw_step, fl_local_step and fl_fedavg each
    against the oracle."""
    torch, P, orc = env["torch"], env["P"], env["orc"]
    r = np.random.default_rng(8)
    sizes = r.integers(1, 9000, 25)
    flags = r.integers(0, 2, sizes.size).astype(np.uint8)
    w = W.make_workload("standalone", sizes, flags, R=5, G=3, A=1,
                        weights=np.array([3, 1, 2], np.float32))
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    dev = synth.buffers.DeviceInputs(w)
    host = synth.buffers.HostInputs(w)
    n = w.n
    _say("standalone n=%d" % n)
    # reduce + per-segment sums of squares
    g_dev = torch.empty(n, dtype=torch.float32, device="cuda")
    ss_dev = torch.empty(w.n_seg, dtype=torch.float32, device="cuda")
    P.fl_shard_reduce(lay, dev.grads[:w.R], w.grad_scale, g_dev, seg_sumsq=ss_dev)
    g_ref = orc.shard_reduce(host.grads[:w.R], w.grad_scale)
    torch.cuda.synchronize()
    assert np.array_equal(g_dev.cpu().numpy().view(np.uint32), g_ref.view(np.uint32))
    H.assert_sumsq("reduce", ss_dev.cpu().numpy(), orc.seg_sumsq(w.seg_offsets, g_ref))
    # AdamW at step 3 from a non-zero state (the reduced gradient as input)
    m0 = (r.standard_normal(n) * 1e-4).astype(np.float32)
    v0 = (np.abs(r.standard_normal(n)) * 1e-7).astype(np.float32)
    dev.m.copy_(torch.from_numpy(m0))
    dev.v.copy_(torch.from_numpy(v0))
    host.m[:] = m0
    host.v[:] = v0
    work_dev = torch.zeros(n, dtype=torch.bfloat16, device="cuda")
    P.fl_adamw_step(lay, w.hp, 3, g_dev, dev.master, dev.m, dev.v, work_dev)
    work_ref = np.zeros(n, np.uint16)
    orc.adamw_step(w.seg_offsets, w.seg_decay, w.hp, 3, g_ref, host.master, host.m, host.v,
                   work_ref)
    torch.cuda.synchronize()
    H.assert_state_parity("adamw", dict(master=dev.master.cpu().numpy(), m=dev.m.cpu().numpy(),
                                        v=dev.v.cpu().numpy(), working=H.to_u16(work_dev)),
                          dict(master=host.master, m=host.m, v=host.v, working=work_ref),
                          bitwise=True)
    # AdamW without the working copy leaves it alone
    P.fl_adamw_step(lay, w.hp, 4, g_dev, dev.master, dev.m, dev.v, None)
    orc.adamw_step(w.seg_offsets, w.seg_decay, w.hp, 4, g_ref, host.master, host.m, host.v)
    torch.cuda.synchronize()
    assert np.array_equal(H.to_u16(work_dev), work_ref)
    H.assert_state_parity("adamw-nowork", dict(master=dev.master.cpu().numpy(),
                                               m=dev.m.cpu().numpy(), v=dev.v.cpu().numpy()),
                          dict(master=host.master, m=host.m, v=host.v), bitwise=True)
    # fused local step
    ss2 = torch.empty(w.n_seg, dtype=torch.float32, device="cuda")
    P.fl_local_step(lay, w.hp, 5, dev.grads[:w.R], w.grad_scale, dev.master, dev.m, dev.v,
                    work_dev, seg_sumsq=ss2)
    orc.adamw_step(w.seg_offsets, w.seg_decay, w.hp, 5, g_ref, host.master, host.m, host.v,
                   work_ref)
    torch.cuda.synchronize()
    H.assert_state_parity("local-step", dict(master=dev.master.cpu().numpy(),
                                             m=dev.m.cpu().numpy(), v=dev.v.cpu().numpy(),
                                             working=H.to_u16(work_dev)),
                          dict(master=host.master, m=host.m, v=host.v, working=work_ref),
                          bitwise=True)
    H.assert_sumsq("local-step", ss2.cpu().numpy(), orc.seg_sumsq(w.seg_offsets, g_ref))
    # FedAvg, in place on the own replica, with fingerprints
    reps_dev = [work_dev if x is None else x for x in dev.replicas]
    reps_ref = [work_ref if x is None else x for x in host.replicas]
    mo_ref, wo_ref = orc.fedavg(reps_ref, w.weights)
    P.fl_fedavg(lay, reps_dev, w.weights, dev.master, work_dev,
                replica_fp=[lay.fingerprint] * w.G)
    torch.cuda.synchronize()
    H.assert_state_parity("fedavg", dict(master=dev.master.cpu().numpy(),
                                         working=H.to_u16(work_dev)),
                          dict(master=mo_ref, working=wo_ref), bitwise=True)
    lay.close()


def test_fused_round_equals_chain(env):
    """fl_round is bitwise the chain fl_local_step x A then fl_fedavg, and the
    fused local step is bitwise fl_shard_reduce then fl_adamw_step."""
    torch, P = env["torch"], env["P"]
    r = np.random.default_rng(9)
    sizes = r.integers(100, 50000, 12)
    flags = r.integers(0, 2, sizes.size).astype(np.uint8)
    w = W.make_workload("chain", sizes, flags, R=3, G=4, A=3, self_group=2,
                        weights=np.array([1, 2, 3, 4], np.float32))
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    a = synth.buffers.DeviceInputs(w)
    b = synth.buffers.DeviceInputs(w)
    c = synth.buffers.DeviceInputs(w)
    H.gpu_round(P, lay, w, a)
    for s in range(w.A):
        P.fl_local_step(lay, w.hp, w.step0 + s, b.grads[s * w.R:(s + 1) * w.R], w.grad_scale,
                        b.master, b.m, b.v, b.working)
        g = torch.empty(w.n, dtype=torch.float32, device="cuda")
        P.fl_shard_reduce(lay, c.grads[s * w.R:(s + 1) * w.R], w.grad_scale, g)
        P.fl_adamw_step(lay, w.hp, w.step0 + s, g, c.master, c.m, c.v, c.working)
    for x in (b, c):
        reps = [x.working if k == w.self_group else x.replicas[k] for k in range(w.G)]
        P.fl_fedavg(lay, reps, w.weights, x.master, x.working)
    torch.cuda.synchronize()
    for x in (b, c):
        for k in ("master", "m", "v", "working"):
            assert torch.equal(getattr(a, k).view(torch.int16 if k == "working" else torch.int32),
                               getattr(x, k).view(torch.int16 if k == "working" else torch.int32)), k
    lay.close()


def test_results_independent_of_grid_and_repeatable(env):
    torch, P = env["torch"], env["P"]
    r = np.random.default_rng(10)
    sizes = r.integers(1, 70000, 40)
    flags = r.integers(0, 2, sizes.size).astype(np.uint8)
    w = W.make_workload("grid", sizes, flags, R=4, G=3, A=2)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    outs = []
    for bpc in (0, 1, 3, 64, 0):
        prev = P.set_blocks_per_cu(bpc)
        try:
            d = synth.buffers.DeviceInputs(w)
            ss = torch.empty(w.A * w.n_seg, dtype=torch.float32, device="cuda")
            H.gpu_round(P, lay, w, d, seg_sumsq=ss)
            torch.cuda.synchronize()
            outs.append([d.master.clone(), d.m.clone(), d.v.clone(), d.working.clone(), ss])
        finally:
            P.set_blocks_per_cu(prev)
    for o in outs[1:]:
        for x, y in zip(outs[0], o):
            assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x.view(torch.int32),
                               y.view(torch.int16) if y.dtype == torch.bfloat16 else y.view(torch.int32))
    lay.close()


def test_special_values(env):
    """NaN, +-inf, subnormal and signed-zero inputs propagate exactly as in the
    oracle."""
    torch, P, orc = env["torch"], env["P"], env["orc"]
    n = 4099
    r = np.random.default_rng(11)
    specials_f32 = np.array([np.nan, np.inf, -np.inf, 0.0, -0.0, 1e-40, -1e-40, 1e-45, 3e38,
                             -3e38, 1.0, -2.5], np.float32)
    specials_bf16 = np.array([0x7FC0, 0xFFC0, 0x7F80, 0xFF80, 0x0000, 0x8000, 0x0001, 0x8001,
                              0x007F, 0x7F7F, 0xFF7F, 0x3F80], np.uint16)
    R, G = 3, 3
    grads = [H.to_u16(torch.from_numpy((r.standard_normal(n) * 1e-3).astype(np.float32))
                      .to(torch.bfloat16)) for _ in range(R)]
    for g in grads:
        pos = r.integers(0, n, 40)
        g[pos] = specials_bf16[r.integers(0, specials_bf16.size, 40)]
    master = (r.standard_normal(n) * 0.02).astype(np.float32)
    master[r.integers(0, n, 40)] = specials_f32[r.integers(0, specials_f32.size, 40)]
    reps = [H.to_u16(torch.from_numpy(master).to(torch.bfloat16)) for _ in range(G)]
    reps[1][r.integers(0, n, 30)] = specials_bf16[r.integers(0, specials_bf16.size, 30)]
    off = np.array([0, 1000, 2500, n], np.int64)
    dec = np.array([1, 0, 1], np.uint8)
    hp = dict(W.ADAMW)
    lay = P.Layout(off, dec)
    tg = [torch.from_numpy(g.view(np.int16)).cuda().view(torch.bfloat16) for g in grads]
    trep = [None] + [torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16) for x in reps[1:]]
    tm = torch.from_numpy(master.copy()).cuda()
    zm = torch.zeros(n, device="cuda")
    zv = torch.zeros(n, device="cuda")
    tw = torch.zeros(n, dtype=torch.bfloat16, device="cuda")
    cfg = P.make_round_cfg(R, G, 2, [1.0, 2.0, 3.0], hp)
    P.fl_round(lay, cfg, tg + tg, trep, tm, zm, zv, tw)
    torch.cuda.synchronize()
    hm, hmm, hv, hw = master.copy(), np.zeros(n, np.float32), np.zeros(n, np.float32), np.zeros(n, np.uint16)
    with np.errstate(all="ignore"):
        orc.round(off, dec, R, G, 2, 0, 1.0 / R, hp, 1, np.array([1, 2, 3], np.float32),
                  grads + grads, [None] + reps[1:], hm, hmm, hv, hw)
    got = dict(master=tm.cpu().numpy(), m=zm.cpu().numpy(), v=zv.cpu().numpy(), working=H.to_u16(tw))
    H.assert_state_parity("specials", got, dict(master=hm, m=hmm, v=hv, working=hw))
    lay.close()


def test_empty_shard(env):
    torch, P = env["torch"], env["P"]
    lay = P.Layout(np.array([0], np.int64), np.zeros(0, np.uint8))
    cfg = P.make_round_cfg(2, 2, 3, [1.0, 1.0], W.ADAMW)
    P.fl_round(lay, cfg, [None] * 6, [None, None], None, None, None, None)
    P.fl_fedavg(lay, [None, None], [1.0, 1.0], None, None)
    P.fl_shard_reduce(lay, [None], 1.0, None)
    torch.cuda.synchronize()
    lay.close()


def test_errors_are_returned_before_any_launch(env):
    torch, P = env["torch"], env["P"]
    n = 5000
    off = np.array([0, 3000, n], np.int64)
    lay = P.Layout(off, np.array([1, 0], np.uint8))
    other = P.Layout(np.array([0, 2999, n], np.int64), np.array([1, 0], np.uint8))
    master = torch.ones(n, device="cuda")
    keep = master.clone()
    m = torch.zeros(n, device="cuda")
    v = torch.zeros(n, device="cuda")
    work = torch.zeros(n, dtype=torch.bfloat16, device="cuda")
    g = [torch.zeros(n, dtype=torch.bfloat16, device="cuda") for _ in range(2)]
    reps = [None, torch.zeros(n, dtype=torch.bfloat16, device="cuda")]
    big = torch.zeros(n + 8, dtype=torch.bfloat16, device="cuda")
    unaligned = big[1:1 + n]

    def status(fn):
        try:
            fn()
        except P.FlError as e:
            return e.status
        return 0

    base = dict(R=2, G=2, A=1, weights=[1.0, 1.0], hp=W.ADAMW)
    cfg = lambda **k: P.make_round_cfg(**{**base, **k})  # noqa: E731
    run = lambda c, gg=g, rr=reps, mm=master: P.fl_round(lay, c, gg, rr, mm, m, v, work)  # noqa: E731
    assert status(lambda: run(cfg(weights=[1.0, -1.0]))) == -1
    assert status(lambda: run(cfg(weights=[0.0, 0.0]))) == -1
    assert status(lambda: run(cfg(hp=dict(W.ADAMW, eps=0.0)))) == -1
    assert status(lambda: run(cfg(hp=dict(W.ADAMW, beta1=1.0)))) == -1
    assert status(lambda: run(cfg(hp=dict(W.ADAMW, lr=float("nan"))))) == -1
    assert status(lambda: run(cfg(step0=0))) == -1
    assert status(lambda: run(cfg(self_group=2))) == -1
    assert status(lambda: run(cfg(R=65))) == -1
    assert status(lambda: run(cfg(max_grad_norm=-1.0))) == -1
    assert status(lambda: run(cfg(max_grad_norm=float("inf")))) == -1
    assert status(lambda: run(cfg(), gg=[g[0], unaligned])) == -2
    assert status(lambda: run(cfg(), rr=[None, None])) == -1
    assert status(lambda: run(cfg(replica_fp=[0, other.fingerprint]))) == -3
    assert status(lambda: P.fl_fedavg(lay, [work, reps[1]], [1, 1], master, work,
                                      replica_fp=[lay.fingerprint, other.fingerprint])) == -3
    assert status(lambda: P.fl_adamw_step(lay, W.ADAMW, 1, m, master, master, v)) == -1
    torch.cuda.synchronize()
    master.copy_(keep)
    assert status(lambda: run(cfg(), mm=master)) == 0
    torch.cuda.synchronize()
    lay.close()
    other.close()


@pytest.mark.parametrize("kind", ["fsdp", "outer", "clip"])
def test_many_rounds_stay_bitwise(env, kind):
    """Twelve consecutive rounds on the same device state (step counter and
    bias corrections advancing, the other groups' replicas fixed), compared
    with the oracle after every round."""
    torch, P, orc = env["torch"], env["P"], env["orc"]
    r = np.random.default_rng(40)
    sizes = r.integers(1, 40_000, 9)
    flags = r.integers(0, 2, sizes.size).astype(np.uint8)
    kw = dict(outer=dict(outer=W.DILOCO_OUTER), clip=dict(max_grad_norm=0.02), fsdp={})[kind]
    w = W.make_workload("rounds_" + kind, sizes, flags, R=4, G=3, A=3, step0=1, **kw)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    dev = B.DeviceInputs(w)
    host = B.HostInputs(w)
    for rnd in range(12):
        step0 = w.step0 + rnd * w.A
        H.gpu_round(P, lay, w, dev, cfg=H.round_cfg(P, w, step0, dev=dev))
        H.oracle_round(orc, W.Workload(**{**w.__dict__, "step0": step0}), host)
        torch.cuda.synchronize()
        got = dict(master=dev.master.cpu().numpy(), m=dev.m.cpu().numpy(),
                   v=dev.v.cpu().numpy(), working=H.to_u16(dev.working))
        H.assert_state_parity("%s round %d" % (kind, rnd), got,
                              dict(master=host.master, m=host.m, v=host.v,
                                   working=host.working), bitwise=True)
        if w.outer is not None:
            assert np.array_equal(dev.buf.cpu().numpy().view(np.uint32), host.buf.view(np.uint32))
    lay.close()


@pytest.mark.parametrize("kind", ["fsdp", "outer"])
def test_resume_from_a_host_checkpoint(env, kind):
    """Checkpoint and resume: after one round the state (master, m, v,
    working; with the outer step also prev and buf) is copied to host memory,
    as a checkpoint would, and loaded into fresh device buffers.  The next
    round from the restored state equals the next round of the uninterrupted
    run bit for bit: a round is a pure function of (state, inputs, step0)."""
    torch, P = env["torch"], env["P"]
    r = np.random.default_rng(44)
    sizes = r.integers(1, 50_000, 7)
    flags = r.integers(0, 2, sizes.size).astype(np.uint8)
    kw = dict(outer=W.DILOCO_OUTER) if kind == "outer" else {}
    w = W.make_workload("resume_" + kind, sizes, flags, R=3, G=3, A=2, step0=5, **kw)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    run = synth.buffers.DeviceInputs(w)
    names = ["master", "m", "v", "working"] + (["prev", "buf"] if kind == "outer" else [])
    H.gpu_round(P, lay, w, run, cfg=H.round_cfg(P, w, w.step0, dev=run))
    torch.cuda.synchronize()
    ckpt = {k: getattr(run, k).cpu().clone() for k in names}   # host copies
    resumed = synth.buffers.DeviceInputs(w)
    for k in names:
        getattr(resumed, k).copy_(ckpt[k])
    step1 = w.step0 + w.A
    H.gpu_round(P, lay, w, run, cfg=H.round_cfg(P, w, step1, dev=run))
    H.gpu_round(P, lay, w, resumed, cfg=H.round_cfg(P, w, step1, dev=resumed))
    torch.cuda.synchronize()
    for k in names:
        a, b = getattr(run, k), getattr(resumed, k)
        view = torch.int16 if k == "working" else torch.int32
        assert torch.equal(a.view(view), b.view(view)), k
    lay.close()
