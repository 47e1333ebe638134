"""GPU edge cases beyond the main parity suite: segment structures that stress
the straddling-tile path, optimiser and weight edge values, two streams
sharing one layout, and capture of fl_round in a HIP graph."""
import numpy as np
import pytest

import harness as H
import synth.buffers as B
from synth import workloads as W

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[gpu-edge]", *a, flush=True)


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


def _parity(env, w, tag, place=None):
    torch, P, orc = env["torch"], env["P"], env["orc"]
    _say(tag, w.describe())
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    dev = B.DeviceInputs(w, place=place)
    ss = torch.full((w.A * w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
    H.gpu_round(P, lay, w, dev, seg_sumsq=ss)
    torch.cuda.synchronize()
    host = B.HostInputs(w)
    ss_ref = H.oracle_round(orc, w, host, want_sumsq=True)
    H.assert_state_parity(tag, _state(dev), dict(master=host.master, m=host.m, v=host.v,
                                                 working=host.working), bitwise=True)
    H.assert_sumsq(tag, ss.cpu().numpy(), ss_ref.reshape(-1))
    lay.close()


@pytest.mark.parametrize("clip,scratch", [(0.0, False), (1e-3, False), (1e-3, True)])
def test_tiles_with_many_segments(env, clip, scratch):
    """Runs of one-element and tiny segments, so single 2048-element tiles
    hold hundreds of segments, between large ones; unclipped, and clipped
    through the sum-of-squares pass or the scratch pass."""
    sizes = [5000] + [1] * 700 + [3, 2, 1] * 100 + [4096, 1, 2047, 2049] + [7] * 300 + [10000]
    r = np.random.default_rng(21)
    flags = r.integers(0, 2, len(sizes)).astype(np.uint8)
    w = W.make_workload("many_segments", sizes, flags, R=3, G=2, A=2, max_grad_norm=clip,
                        clip_scratch=scratch)
    _parity(env, w, "many_segments clip=%g scratch=%s" % (clip, scratch))


@pytest.mark.parametrize("hp,step0", [
    (dict(lr=3e-4, beta1=0.0, beta2=0.0, eps=1e-8, weight_decay=0.1), 1),
    (dict(lr=3e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.0), 1_000_000),
    (dict(lr=0.5, beta1=0.99, beta2=0.999, eps=1e-3, weight_decay=1.5), 2),
    (dict(lr=0.0, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1), 7),
])
def test_optimiser_edge_values(env, hp, step0):
    r = np.random.default_rng(22)
    sizes = r.integers(1, 30000, 10)
    flags = r.integers(0, 2, sizes.size).astype(np.uint8)
    w = W.make_workload("hp_edges", sizes, flags, R=2, G=3, A=2, hp=hp, step0=step0,
                        weights=np.array([0.0, 2.0, 0.0], np.float32), self_group=1)
    _parity(env, w, "hp %s step0 %d" % (hp, step0))


def test_two_streams_share_a_layout(env):
    """Two rounds on two streams, one layout: the second stream's call waits
    for the first call's kernels and then reuses the layout's workspace;
    both match the oracle."""
    torch, P, orc = env["torch"], env["P"], env["orc"]
    r = np.random.default_rng(23)
    sizes = r.integers(1, 200000, 30)
    flags = r.integers(0, 2, sizes.size).astype(np.uint8)
    wa = W.make_workload("stream_a", sizes, flags, R=4, G=2, A=3, seed=1)
    wb = W.make_workload("stream_b", sizes, flags, R=4, G=2, A=3, seed=2)
    lay = P.Layout(wa.seg_offsets, wa.seg_decay)
    da, db = B.DeviceInputs(wa), B.DeviceInputs(wb)
    torch.cuda.synchronize()
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    ssa = torch.empty(wa.A * wa.n_seg, dtype=torch.float32, device="cuda")
    ssb = torch.empty(wb.A * wb.n_seg, dtype=torch.float32, device="cuda")
    with torch.cuda.stream(sa):
        H.gpu_round(P, lay, wa, da, seg_sumsq=ssa)
    with torch.cuda.stream(sb):
        H.gpu_round(P, lay, wb, db, seg_sumsq=ssb)
    torch.cuda.synchronize()
    for w, d, ss in ((wa, da, ssa), (wb, db, ssb)):
        host = B.HostInputs(w)
        ref = H.oracle_round(orc, w, host, want_sumsq=True)
        H.assert_state_parity(w.name, _state(d), dict(master=host.master, m=host.m, v=host.v,
                                                      working=host.working), bitwise=True)
        H.assert_sumsq(w.name, ss.cpu().numpy(), ref.reshape(-1))
    lay.close()


def test_round_captured_in_a_hip_graph(env):
    """fl_round (without per-segment sums it allocates nothing) captured once
    and replayed three times, with eager work and synchronisation between
    replays; every replay equals the eager result of the same round."""
    torch, P = env["torch"], env["P"]
    r = np.random.default_rng(24)
    sizes = r.integers(1, 60000, 12)
    flags = r.integers(0, 2, sizes.size).astype(np.uint8)
    w = W.make_workload("graph", sizes, flags, R=4, G=3, A=2)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    eager = B.DeviceInputs(w)
    graphed = B.DeviceInputs(w)
    cfg = P.make_round_cfg(w.R, w.G, w.A, w.weights, w.hp, self_group=w.self_group,
                           grad_scale=w.grad_scale, step0=w.step0)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    # the capture records the same kernel launches; it does not run them
    snapshot = [t.clone() for t in (graphed.master, graphed.m, graphed.v, graphed.working)]
    with torch.cuda.graph(g, stream=s):
        P.fl_round(lay, cfg, graphed.grads, graphed.replicas, graphed.master, graphed.m,
                   graphed.v, graphed.working)
    torch.cuda.synchronize()
    for t, snap in zip((graphed.master, graphed.m, graphed.v, graphed.working), snapshot):
        assert torch.equal(t.view(torch.int16), snap.view(torch.int16)), "capture ran kernels"
    for rep in range(3):
        P.fl_round(lay, cfg, eager.grads, eager.replicas, eager.master, eager.m, eager.v,
                   eager.working)
        junk = torch.randn(1 << 20, device="cuda").sum()  # unrelated eager work
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name in ("master", "m", "v", "working"):
            a = getattr(eager, name)
            b = getattr(graphed, name)
            assert torch.equal(a.view(torch.int16), b.view(torch.int16)), \
                "replay %d differs in %s" % (rep, name)
        del junk
    lay.close()


def test_round_with_scheduled_learning_rates(env):
    """Each local step of a round uses its own scheduled learning rate (cosine
    decay with warm-up); the library's and the oracle's schedules are computed
    separately and agree bitwise."""
    torch, P, orc = env["torch"], env["P"], env["orc"]
    r = np.random.default_rng(25)
    sizes = r.integers(1, 50000, 9)
    flags = r.integers(0, 2, sizes.size).astype(np.uint8)
    w = W.make_workload("sched", sizes, flags, R=3, G=2, A=4, step0=5)
    T, Wu = 64, 7
    lib_lrs = [P.lr_cosine(w.step0 + a, T, Wu, w.hp["lr"]) for a in range(w.A)]
    orc_lrs = [orc.lr_cosine(w.step0 + a, T, Wu, w.hp["lr"]) for a in range(w.A)]
    assert np.array_equal(np.float32(lib_lrs), np.float32(orc_lrs))
    assert len(set(lib_lrs)) == w.A
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    dev = B.DeviceInputs(w)
    cfg = P.make_round_cfg(w.R, w.G, w.A, w.weights, w.hp, self_group=w.self_group,
                           grad_scale=w.grad_scale, step0=w.step0, step_lr=lib_lrs)
    ss = torch.empty(w.A * w.n_seg, dtype=torch.float32, device="cuda")
    H.gpu_round(P, lay, w, dev, seg_sumsq=ss, cfg=cfg)
    torch.cuda.synchronize()
    host = B.HostInputs(w)
    ss_ref = orc.round(w.seg_offsets, w.seg_decay, w.R, w.G, w.A, w.self_group, w.grad_scale,
                       w.hp, w.step0, w.weights, host.grads, host.replicas, host.master, host.m,
                       host.v, host.working, want_sumsq=True, step_lr=orc_lrs)
    H.assert_state_parity("sched", _state(dev), dict(master=host.master, m=host.m, v=host.v,
                                                     working=host.working), bitwise=True)
    H.assert_sumsq("sched", ss.cpu().numpy(), ss_ref.reshape(-1))
    bad = P.make_round_cfg(w.R, w.G, w.A, w.weights, w.hp, step_lr=[1e-3, -1.0, 1e-3, 1e-3])
    with pytest.raises(P.FlError):
        H.gpu_round(P, lay, w, dev, cfg=bad)
    lay.close()


def test_binding_rejects_mismatched_tensors(env):
    """Tensors of the wrong length or element size, and lists of the wrong
    length, are refused on the host before anything is enqueued; a list
    shorter than the configuration asks for reaches the library as NULL
    entries, which it rejects."""
    torch, P = env["torch"], env["P"]
    n = 4099
    lay = P.Layout(np.array([0, 1000, n], np.int64), np.array([1, 0], np.uint8))
    f32 = lambda k=n: torch.zeros(k, dtype=torch.float32, device="cuda")  # noqa: E731
    bf = lambda k=n: torch.zeros(k, dtype=torch.bfloat16, device="cuda")  # noqa: E731
    master, m, v, work = f32(), f32(), f32(), bf()
    keep = master.clone()
    grads = [bf(), bf()]
    cfg = P.make_round_cfg(2, 2, 1, [1.0, 1.0], W.ADAMW)
    run = lambda **k: P.fl_round(lay, cfg, k.get("g", grads), k.get("r", [None, bf()]),  # noqa: E731
                                 k.get("p", master), m, v, work, seg_sumsq=k.get("ss"))
    with pytest.raises(ValueError, match="elements"):
        run(p=f32(n - 1))
    with pytest.raises(ValueError, match="byte elements"):
        run(g=[grads[0], f32()])
    with pytest.raises(ValueError, match="entries"):
        run(g=grads + [bf()])
    with pytest.raises(ValueError, match="elements"):
        run(ss=f32(lay.n_seg + 1))
    with pytest.raises(ValueError, match="contiguous"):
        run(p=torch.zeros(2 * n, device="cuda")[::2])
    with pytest.raises(P.FlError) as e:
        run(g=grads[:1])
    assert e.value.status == -1
    torch.cuda.synchronize()
    assert torch.equal(master, keep), "a refused call changed the state"
    lay.close()


@pytest.mark.parametrize("kind", ["clip", "clip-scratch", "hsdp", "hsdp-recv", "outer"])
def test_every_path_is_independent_of_the_launch_shape(env, kind):
    """The same round under the default launch shapes and three forced ones
    (1, 3 and 7 workgroups per CU for every pass) gives the same bits: state,
    outer state and per-segment sums."""
    torch, P = env["torch"], env["P"]
    r = np.random.default_rng(26)
    sizes = r.integers(1, 90_000, 17)
    flags = r.integers(0, 2, sizes.size).astype(np.uint8)
    kw = dict(clip=dict(max_grad_norm=0.01), hsdp=dict(H=3, replica=2),
              outer=dict(outer=W.DILOCO_OUTER))
    kw["clip-scratch"] = dict(max_grad_norm=0.01, clip_scratch=True)
    kw["hsdp-recv"] = dict(H=2, replica=1, hsdp_member=False, max_grad_norm=0.01)
    w = W.make_workload("shape_" + kind, sizes, flags, R=6, G=3, A=2, step0=4, **kw[kind])
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    results = []
    prev = P.set_blocks_per_cu(0)
    try:
        for bpc in (0, 1, 3, 7):
            P.set_blocks_per_cu(bpc)
            dev = B.DeviceInputs(w)
            ss = torch.full((w.A * w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
            H.gpu_round(P, lay, w, dev, seg_sumsq=ss)
            torch.cuda.synchronize()
            keep = [dev.master, dev.m, dev.v, dev.working, ss]
            if w.outer is not None:
                keep += [dev.prev, dev.buf]
            results.append([t.clone() for t in keep])
            del dev
    finally:
        P.set_blocks_per_cu(prev)
    for bpc, res in zip((1, 3, 7), results[1:]):
        for a, b in zip(results[0], res):
            assert torch.equal(a.view(torch.int16), b.view(torch.int16)), \
                "%s differs at %d workgroups per CU" % (kind, bpc)
    lay.close()


def test_hundreds_of_thousands_of_segments(env):
    """300,000 segments of 1-8 elements: every tile straddles segments, and
    the finalize kernels fold 300,000 per-segment sums (clipped round, so the
    whole-shard total too)."""
    r = np.random.default_rng(27)
    sizes = r.integers(1, 9, 300_000)
    flags = r.integers(0, 2, sizes.size).astype(np.uint8)
    w = W.make_workload("many_many_segments", sizes, flags, R=2, G=2, A=2, max_grad_norm=0.01)
    _parity(env, w, "300k segments")


def _chain_of_calls(env, lay, w, d, ss):
    """The round of w as the chain of standalone calls on the inputs d:
    fl_local_step with per-segment sums (each pass followed by its finalize
    kernel) A times, then fl_fedavg, or fl_fedopt with an outer step."""
    P = env["P"]
    for s in range(w.A):
        P.fl_local_step(lay, w.hp, w.step0 + s, d.grads[s * w.R:(s + 1) * w.R], w.grad_scale,
                        d.master, d.m, d.v, d.working, seg_sumsq=ss[s * w.n_seg:(s + 1) * w.n_seg])
    reps = [d.working if k == w.self_group else d.replicas[k] for k in range(w.G)]
    if w.outer is not None:
        P.fl_fedopt(lay, reps, w.weights, w.outer, d.prev, d.buf, d.master, d.working)
    else:
        P.fl_fedavg(lay, reps, w.weights, d.master, d.working)


@pytest.mark.parametrize("sizes,outer", [
    ([1 << 20], False),                                          # one segment (the tiny round's shape)
    ([300000, 17, 2047, 2049, 1 << 20, 5, 9, 70000], False),    # 8 segments
    ([300000, 17, 2047, 2049, 1 << 20, 5, 9, 70000], True),     # the same with the outer step
    ([1024 * 2048, 3], False),                                   # a segment of exactly 1024 tiles
    ([1000, 1, 2, 3, 4, 5, 6, 7, 5000], False),                  # 9 segments: finalize kernels
    ([1025 * 2048, 5], False),                                   # a two-chunk segment: the same
])
def test_carried_finalize_matches_the_chain_of_calls(env, sizes, outer):
    """Where the round leaves each step's finalize to its next kernel (at
    most 8 segments, each one finalize chunk), the per-segment sums and every
    output are bitwise those of the chain of standalone calls, whose passes
    are each followed by the finalize kernel; both equal the oracle."""
    torch, P = env["torch"], env["P"]
    flags = (np.arange(len(sizes)) % 2).astype(np.uint8)
    kw = dict(outer=dict(lr=0.7, momentum=0.9, nesterov=True)) if outer else {}
    w = W.make_workload("carry", sizes, flags, R=4, G=2, A=3, seed=5, **kw)
    _say(w.describe())
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    d0, d1 = B.DeviceInputs(w), B.DeviceInputs(w)
    s0 = torch.full((w.A * w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
    s1 = torch.full((w.A * w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    H.gpu_round(P, lay, w, d0, seg_sumsq=s0)
    _chain_of_calls(env, lay, w, d1, s1)
    torch.cuda.synchronize()
    a, b = _state(d0), _state(d1)
    a["ss"], b["ss"] = s0.cpu().numpy(), s1.cpu().numpy()
    for k in a:
        u = np.uint16 if k == "working" else np.uint32
        assert np.array_equal(np.asarray(a[k]).view(u), np.asarray(b[k]).view(u)), k
    host = B.HostInputs(w)
    ref = H.oracle_round(env["orc"], w, host, want_sumsq=True)
    H.assert_state_parity("carry", a, dict(master=host.master, m=host.m, v=host.v,
                                           working=host.working), bitwise=True)
    H.assert_sumsq("carry", a["ss"], ref.reshape(-1))
    lay.close()


@pytest.mark.parametrize("member,clip", [(True, 0.0), (False, 0.0), (True, 1e-3), (False, 1e-3)])
def test_carried_finalize_in_hsdp_rounds(env, member, clip):
    """FL+HSDP rounds (H = 2) on a layout whose finalize the round carries:
    into the next step's kernel, then into FedAvg (member) or the broadcast
    receive (receiver); clipped rounds use the finalize kernels instead.
    Every output against the oracle."""
    sizes = [300000, 17, 2047, 2049, 1 << 20, 5]
    flags = (np.arange(len(sizes)) % 2).astype(np.uint8)
    w = W.make_workload("carry_hsdp", sizes, flags, R=3, G=2, A=3, H=2, replica=1,
                        hsdp_member=member, max_grad_norm=clip, seed=6)
    _parity(env, w, "carry_hsdp member=%s clip=%g" % (member, clip))


def test_grad_sumsq_on_two_streams(env):
    """fl_grad_sumsq on two streams in turn, one layout (the second waits for
    the first's kernels and reuses the workspace): the whole-shard totals and
    per-segment sums are bitwise equal and equal the oracle's within
    tolerance."""
    torch, P, orc = env["torch"], env["P"], env["orc"]
    sizes = [50000, 3, 1 << 19, 77777]
    w = W.make_workload("sumsq_streams", sizes, [1, 0, 1, 1], R=3, G=2, A=1, seed=9)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    d = B.DeviceInputs(w)
    torch.cuda.synchronize()
    outs = []
    for s in (torch.cuda.Stream(), torch.cuda.Stream()):
        tot = torch.full((1,), -1.0, dtype=torch.float64, device="cuda")
        ss = torch.full((w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
        with torch.cuda.stream(s):
            P.fl_grad_sumsq(lay, d.grads[:w.R], w.grad_scale, tot, ss)
        outs.append((tot, ss))
    torch.cuda.synchronize()
    (t0, s0), (t1, s1) = outs
    assert t0.cpu().numpy().view(np.uint64)[0] == t1.cpu().numpy().view(np.uint64)[0]
    assert np.array_equal(s0.cpu().numpy().view(np.uint32), s1.cpu().numpy().view(np.uint32))
    host = B.HostInputs(w)
    g = orc.shard_reduce(host.grads[:w.R], w.grad_scale)
    ref_ss = orc.seg_sumsq(w.seg_offsets, g)
    H.assert_sumsq("sumsq_streams segs", s0.cpu().numpy(), ref_ss)
    H.assert_sumsq("sumsq_streams", t0.cpu().numpy(), np.array([orc.total_sumsq(g)]))
    lay.close()


@pytest.mark.parametrize("clip", [0.0, 1e-3])
def test_multi_chunk_finalize_against_oracle(env, clip):
    """Segments of exactly 1024 tiles (one finalize chunk), 1025 tiles (two
    chunks, so the per-segment fold of chunk sums runs) and about 5 M
    elements (three chunks), between short ones; every per-segment sum of
    squares against the oracle, unclipped and clipped."""
    sizes = [1024 * 2048, 1025 * 2048, 5_000_003, 7, 300, 1, 4096]
    flags = np.array([1, 1, 0, 1, 0, 1, 1], np.uint8)
    w = W.make_workload("multi_chunk", sizes, flags, R=2, G=2, A=2, max_grad_norm=clip, seed=12)
    _parity(env, w, "multi_chunk clip=%g" % clip)


def test_phase_events_with_null_entries(env):
    """Phase events only before the first local step, before FedAvg and after
    it (NULL entries between them): the round's outputs equal an untimed
    round's bit for bit, and the three events bracket the steps and
    FedAvg."""
    torch, P = env["torch"], env["P"]
    w = W.make_workload("events", [300000, 17, 5000], [1, 0, 1], R=3, G=2, A=3, seed=4)
    lay = P.Layout(w.seg_offsets, w.seg_decay)
    d0, d1 = B.DeviceInputs(w), B.DeviceInputs(w)
    s0 = torch.full((w.A * w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
    s1 = torch.full((w.A * w.n_seg,), -1.0, dtype=torch.float32, device="cuda")
    ev = P.HipEvents(3, P.HIP_EVENT_DISABLE_SYSTEM_FENCE)
    hs = [ev.handles[0], None, None, ev.handles[1], ev.handles[2]]
    torch.cuda.synchronize()
    H.gpu_round(P, lay, w, d0, seg_sumsq=s0, phase_events=hs)
    H.gpu_round(P, lay, w, d1, seg_sumsq=s1)
    torch.cuda.synchronize()
    a, b = _state(d0), _state(d1)
    a["ss"], b["ss"] = s0.cpu().numpy(), s1.cpu().numpy()
    for k in a:
        u = np.uint16 if k == "working" else np.uint32
        assert np.array_equal(np.asarray(a[k]).view(u), np.asarray(b[k]).view(u)), k
    assert ev.elapsed_ms(0, 1) > 0 and ev.elapsed_ms(1, 2) > 0
    ev.close()
    lay.close()


def test_separate_arrays_allocates_and_frees_exact_blocks(env):
    """separate_arrays gives each array a device allocation of its own, wraps it
    without a copy, and frees it with the tensor; a round on such arrays is
    bitwise equal to the oracle."""
    import gc

    torch, P = env["torch"], env["P"]
    _say("separate_arrays: allocation, release, round")
    n = 64 << 20
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    free0 = torch.cuda.mem_get_info()[0]
    ts = P.separate_arrays(n, [torch.float32, torch.bfloat16, torch.bfloat16])
    assert [t.dtype for t in ts] == [torch.float32, torch.bfloat16, torch.bfloat16]
    assert all(t.is_cuda and t.numel() == n and t.is_contiguous() for t in ts)
    assert len({t.untyped_storage().data_ptr() for t in ts}) == 3
    assert all(t.data_ptr() % 256 == 0 for t in ts)
    spans = sorted((t.data_ptr(), t.data_ptr() + n * t.element_size()) for t in ts)
    assert all(a[1] <= b[0] for a, b in zip(spans, spans[1:]))
    torch.cuda.synchronize()
    assert free0 - torch.cuda.mem_get_info()[0] >= 6 * n       # 8n bytes, to reporting slack
    ts[1].fill_(1.5)
    ts[0].zero_()
    ts[2].zero_()
    assert float(ts[1].float().sum()) == 1.5 * n and float(ts[0].abs().sum()) == 0.0
    del ts
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()      # what the checks above took from torch's allocator
    assert free0 - torch.cuda.mem_get_info()[0] < 2 * n    # the blocks were freed
    assert P.separate_arrays(0, [torch.float32])[0].numel() == 0
    r = np.random.default_rng(71)
    sizes = r.integers(1, 90000, 40)
    w = W.make_workload("placed", sizes, r.integers(0, 2, sizes.size).astype(np.uint8),
                        R=4, G=2, A=2)
    _parity(env, w, "placed", place=P.separate_arrays)
    torch.cuda.empty_cache()
