"""The full-size checks' methods, validated on the CPU on shards small enough
for the oracle to run whole:
  * running the oracle on sampled elements only (with the compacted layout
    and, for clipping, the streamed whole-shard sums of squares) gives exactly
    the whole-shard oracle's values at those elements;
  * the chunked whole-shard comparison of the full-size GPU tests (chunks
    split into per-thread sub-spans with their own layouts) accepts the
    one-pass oracle's result for every round kind and rejects a single
    changed element."""
import numpy as np
import pytest

import harness as H
import oracle
import synth.buffers as B
from synth import workloads as W


@pytest.fixture(scope="module")
def orc():
    import oracle

    return oracle.Oracle()


def _workload(clip, H_=1, outer=None):
    r = np.random.default_rng(31)
    sizes = r.integers(1, 90_000, 40)
    flags = r.integers(0, 2, sizes.size).astype(np.uint8)
    return W.make_workload("sampled_clip%g" % clip, sizes, flags, R=3, G=3, A=3, seed=4,
                           distinct_grads=True, max_grad_norm=clip, outer=outer, H=H_)


@pytest.mark.parametrize("clip,outer", [(0.0, None), (1e-3, None), (1e-3, W.DILOCO_OUTER)])
def test_sampled_oracle_matches_whole_shard(orc, clip, outer):
    w = _workload(clip, outer=outer)
    whole = B.HostInputs(w)
    ss_whole = H.oracle_round(orc, w, whole, want_sumsq=True)
    idx, full = W.sample_indices(w, n_random=5000)
    totals = H.clip_totals(orc, w, chunk=100_000) if clip > 0 else None
    if clip > 0:
        coefs = [orc.clip_coef(t, clip) for t in totals]
        assert all(0.0 < c < 1.0 for c in coefs), "clipping inactive: the case tests nothing"
    host = B.HostInputs(w, idx)
    off, dec, cmap = H.compact_layout(w, idx, full)
    ss = H.oracle_round(orc, w, host, seg_off=off, seg_decay=dec, want_sumsq=True,
                        clip_totals=totals)
    for name in ("master", "m", "v", "working"):
        assert np.array_equal(getattr(host, name), getattr(whole, name)[idx]), name
    if outer is not None:
        assert np.array_equal(host.prev, whole.prev[idx])
        assert np.array_equal(host.buf, whole.buf[idx])
    for s, cs in cmap.items():
        assert np.array_equal(ss[:, cs], ss_whole[:, s])
    if clip > 0:
        # the sampled run without the whole-shard totals would clip differently
        host2 = B.HostInputs(w, idx)
        H.oracle_round(orc, w, host2, seg_off=off, seg_decay=dec)
        assert not np.array_equal(host2.master, host.master)


@pytest.mark.parametrize("threads", [2, 5])
def test_oracle_in_concurrent_chunks_matches_one_pass(orc, threads):
    """The oracle run as contiguous chunks on several threads at once (as the
    benchmark's CPU baseline runs it) gives the whole-shard pass's state bit
    for bit: the path is elementwise, so the thread count changes nothing."""
    from concurrent.futures import ThreadPoolExecutor

    w = _workload(0.0, outer=W.DILOCO_OUTER)
    whole = B.HostInputs(w)
    H.oracle_round(orc, w, whole)
    bounds = np.linspace(0, w.n, threads + 1).astype(np.int64)
    parts = []
    for t in range(threads):
        lo, hi = int(bounds[t]), int(bounds[t + 1])
        inner = w.seg_offsets[(w.seg_offsets > lo) & (w.seg_offsets < hi)]
        off = np.concatenate([[lo], inner, [hi]]).astype(np.int64) - lo
        first = int(np.searchsorted(w.seg_offsets, lo, side="right")) - 1
        parts.append((B.HostInputs(w, span=(lo, hi)), off, w.seg_decay[first:first + off.size - 1]))
    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(lambda p: H.oracle_round(orc, w, p[0], seg_off=p[1], seg_decay=p[2]), parts))
    for name in ("master", "m", "v", "working", "prev", "buf"):
        got = np.concatenate([getattr(p[0], name) for p in parts])
        assert np.array_equal(got, getattr(whole, name)), name


def _whole_shard_case(w, chunk, threads, plant=None):
    orc = oracle.Oracle()
    full = B.HostInputs(w)
    ss_full = H.oracle_round(orc, w, full, want_sumsq=True)
    if plant is not None:
        k, i = plant
        arr = getattr(full, k)
        arr[i] = arr[i] + (arr[i] * 1e-6 if k != "working" else 1)

    def state(k, lo, hi):
        return getattr(full, k)[lo:hi]

    return H.whole_shard_parity(orc, w, state, ss_full.astype(np.float32),
                                lambda lo, hi: B.HostInputs(w, span=(lo, hi)), chunk=chunk,
                                threads=threads)


@pytest.mark.parametrize("kind", ["fsdp", "hsdp_member", "hsdp_recv", "outer"])
def test_whole_shard_method_matches_one_pass(kind):
    """The full-size GPU tests' comparison (chunks of the shard, each split
    into per-thread sub-spans with their own layouts, per-segment sums
    accumulated across pieces) accepts the one-pass oracle's own result, for
    every round kind, with chunks and sub-spans that cut segments."""
    sizes = [3000, 17, 5000, 1, 40000, 777]
    dec = [1, 0, 1, 1, 0, 1]
    wts = np.array([1, 2, 3], np.float32)
    extra = dict(hsdp_member=dict(H=2, replica=1), hsdp_recv=dict(H=2, replica=0, hsdp_member=False),
                 outer=dict(outer=W.DILOCO_OUTER), fsdp={})[kind]
    w = W.make_workload("t_" + kind, sizes, dec, R=3, G=3, A=3, weights=wts, **extra)
    worst = _whole_shard_case(w, chunk=10007, threads=5)
    assert worst["master"] == 0 and worst["working_ulp"] == 0


def test_whole_shard_method_clipped_with_streamed_totals():
    """A clipped round compared chunk by chunk against the oracle given the
    streamed whole-shard totals gives the one-pass clipped oracle's bits."""
    w = W.make_workload("t_clip", [3000, 17, 5000, 1, 40000, 777], [1, 0, 1, 1, 0, 1], R=3, G=3,
                        A=3, weights=np.array([1, 2, 3], np.float32), max_grad_norm=0.05)
    orc = oracle.Oracle()
    full = B.HostInputs(w)
    ss_full = H.oracle_round(orc, w, full, want_sumsq=True)
    totals = H.clip_totals(orc, w, chunk=9000)

    def state(k, lo, hi):
        return getattr(full, k)[lo:hi]

    worst = H.whole_shard_parity(orc, w, state, ss_full.astype(np.float32),
                                 lambda lo, hi: B.HostInputs(w, span=(lo, hi)), chunk=10007,
                                 threads=4, clip_totals=totals)
    assert worst["master"] == 0


@pytest.mark.parametrize("plant", [("master", 44000), ("m", 0), ("v", 48794), ("working", 20014)])
def test_whole_shard_method_catches_one_element(plant):
    """One changed element anywhere (first, last, chunk boundary, interior)
    fails the comparison."""
    w = W.make_workload("t_plant", [3000, 17, 5000, 1, 40000, 777], [1, 0, 1, 1, 0, 1], R=2, G=2,
                        A=2, weights=np.array([1, 1], np.float32))
    with pytest.raises(AssertionError):
        _whole_shard_case(w, chunk=10007, threads=3, plant=plant)


def test_oracle_binding_concurrent_calls_keep_their_arrays():
    """Concurrent oracle rounds (as the whole-shard comparison runs them, one
    per host thread) each with its own clip totals and step learning rates
    give the same results as the same calls made one at a time: the binding
    must keep every call's scalar arrays alive until that call returns."""
    from concurrent.futures import ThreadPoolExecutor

    w = W.make_workload("t_conc", [4096] * 8, [1] * 8, R=2, G=2, A=3,
                        weights=np.array([1, 1], np.float32), max_grad_norm=0.02)
    orc = oracle.Oracle()
    base = B.HostInputs(w)
    jobs = []
    for j in range(64):
        tot = [1e-3 * (j + 1), 2e-3 * (j + 1), 3e-3 * (j + 1)]
        lrs = [1e-4 * (1 + (j % 5)), 2e-4, 3e-4]
        jobs.append((tot, lrs))

    def one(job):
        tot, lrs = job
        h = B.HostView(base, 0, w.n)
        h.master, h.m, h.v, h.working = (base.master.copy(), base.m.copy(), base.v.copy(),
                                         base.working.copy())
        oracle.workload_round(orc, w, h, clip_totals=[float(x) for x in tot],
                              step_lr=[float(x) for x in lrs])
        return h.master

    seq = [one(j) for j in jobs]
    with ThreadPoolExecutor(16) as ex:
        par = list(ex.map(one, jobs))
    for a, b in zip(seq, par):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
