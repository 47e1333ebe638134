"""The sampled full-size check, validated on the CPU: on a shard small enough
for the oracle to run whole, running it on the sampled elements only (with the
compacted layout and, for clipping, the streamed whole-shard sums of squares)
gives exactly the whole-shard oracle's values at those elements."""
import numpy as np
import pytest

import harness as H
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
