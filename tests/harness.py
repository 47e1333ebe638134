"""Helpers shared by the GPU parity tests, smoke() and bench.py.

Inputs come only from the synth generator (device fills for the GPU side,
host values for the oracle side); expected values come only from the oracle.
"""
import numpy as np

from synth.buffers import DeviceInputs, HostInputs, gather_f32, gather_u16, to_u16  # noqa: F401
from synth import host_fill
from synth.workloads import Workload

TOL_F32_REL = 2e-6      # max relative error on fp32 master, m, v
TOL_BF16_ULP = 1        # max distance in bf16 ulps on working copies
TOL_SUMSQ_REL = 1e-5    # per-segment sums of squares vs the double oracle


def compact_layout(w: Workload, idx, full_segments=()):
    """Layout over sampled elements: each full segment's elements (all of them
    must be in idx, consecutively) form one compact segment; every other
    sampled element is a one-element segment with its own segment's flag.
    Returns (offsets, decay, {full segment id: compact segment id})."""
    seg_of = np.searchsorted(w.seg_offsets, idx, side="right") - 1
    full = set(int(s) for s in full_segments)
    off = [0]
    dec = []
    cmap = {}
    j = 0
    n = idx.size
    while j < n:
        s = int(seg_of[j])
        if s in full and idx[j] == w.seg_offsets[s]:
            k = j + int(w.seg_offsets[s + 1] - w.seg_offsets[s])
            assert np.array_equal(idx[j:k], np.arange(w.seg_offsets[s], w.seg_offsets[s + 1]))
            cmap[s] = len(dec)
            off.append(k)
            dec.append(w.seg_decay[s])
            j = k
        else:
            off.append(j + 1)
            dec.append(w.seg_decay[s])
            j += 1
    return np.array(off, np.int64), np.array(dec, np.uint8), cmap


def oracle_round(orc, w: Workload, host: HostInputs, seg_off=None, seg_decay=None,
                 want_sumsq=False, clip_totals=None, step_lr=None):
    """The oracle round of workload w in place on host arrays (see
    oracle.workload_round)."""
    import oracle

    return oracle.workload_round(orc, w, host, seg_off=seg_off, seg_decay=seg_decay,
                                 want_sumsq=want_sumsq, clip_totals=clip_totals,
                                 step_lr=step_lr)


def clip_totals(orc, w: Workload, chunk=1 << 24, say=None, fill=None):
    """Whole-shard sum of squares of each local step's reduced gradient, in
    index order, one chunk of regenerated peer gradients at a time (for a
    clipped round whose oracle sees only part of the shard).  fill(spec, lo,
    k): the k values from index lo (default: the host generator)."""
    assert w.H == 1, "the FL+HSDP clip norm is that of the replica average"
    fill = host_fill if fill is None else fill
    steps = [tuple(w.grad_index[a * w.R:(a + 1) * w.R]) for a in range(w.A)]
    done = {}
    for key in dict.fromkeys(steps):
        acc = 0.0
        for c, lo in enumerate(range(0, w.n, chunk)):
            k = min(chunk, w.n - lo)
            acc = orc.grad_total([fill(w.grad_specs[j], lo, k) for j in key],
                                 w.grad_scale, acc)
            if say is not None and c % 16 == 15:
                say("clip total: %d of %d elements" % (lo + k, w.n))
        done[key] = acc
    return [done[key] for key in steps]


def _bits_equal(got, ref):
    """Every element bitwise equal (a fast whole-array check; NaNs compare as
    bits here, the detailed comparison below tolerates payload differences)."""
    g, r = np.asarray(got), np.asarray(ref)
    if g.shape != r.shape or g.dtype.itemsize != r.dtype.itemsize:
        return False
    u = np.uint32 if g.dtype.itemsize == 4 else np.uint16
    return bool(np.array_equal(g.view(u), r.view(u)))


def assert_state_parity_fast(tag, gpu, ref):
    """assert_state_parity(bitwise=True) with a fast path: arrays that are
    bitwise equal (the expected case) are not examined further; any other
    array goes through the detailed comparison, which reports the errors and
    raises unless only NaN payloads differ."""
    slow = {k: gpu[k] for k in ref if not _bits_equal(gpu[k], ref[k])}
    errs = {k: 0.0 for k in ("master", "m", "v") if k in ref}
    if "working" in ref:
        errs["working_ulp"] = 0
    if slow:
        errs.update(assert_state_parity(tag, slow, {k: ref[k] for k in slow}, bitwise=True))
    return errs


def whole_shard_parity(orc, w: Workload, state, ss_gpu, inputs, chunk=1 << 26, threads=None,
                       clip_totals=None, say=None):
    """Compare every element of a GPU round's result with the oracle.

    state(name, lo, hi) -> host copy of the GPU's array `name` (master, m, v,
    working; prev and buf with an outer step) over elements lo..hi-1;
    ss_gpu: the GPU's A x n_seg sums of squares; inputs(lo, hi) -> the
    HostInputs of that span.  Each chunk of `chunk` elements is split into
    one contiguous sub-span per thread, each with the segments it holds as
    its own layout, and the unchanged oracle runs on every sub-span (ctypes
    releases the GIL; the oracle is elementwise, so sub-spans give the whole
    shard's values).  While the oracle threads work on one chunk, the calling
    thread fetches the next chunk's inputs.  master, m, v and working (and
    the outer state) must be bitwise equal; each segment's sum of squares is
    the sum of its pieces' oracle sums in index order, within TOL_SUMSQ_REL.
    Returns the largest errors seen."""
    from concurrent.futures import ThreadPoolExecutor

    from synth import host_threads
    from synth.buffers import HostView

    T = threads or host_threads()
    seg_acc = np.zeros((w.A, w.n_seg), np.float64)
    worst = {}
    starts = list(range(0, w.n, chunk))

    def run(job):
        view, off, dec, first = job
        return first, oracle_round(orc, w, view, seg_off=off, seg_decay=dec, want_sumsq=True,
                                   clip_totals=clip_totals)

    with ThreadPoolExecutor(T) as ex:
        nxt = inputs(starts[0], min(w.n, starts[0] + chunk)) if starts else None
        for c, lo in enumerate(starts):
            hi = min(w.n, lo + chunk)
            host, nxt = nxt, None
            bounds = np.linspace(0, hi - lo, T + 1).astype(np.int64)
            jobs = []
            for t in range(T):
                a, b = int(bounds[t]), int(bounds[t + 1])
                if b > a:
                    off, dec, first = w.span_layout(lo + a, lo + b)
                    jobs.append((HostView(host, a, b), off, dec, first))
            futs = [ex.submit(run, j) for j in jobs]
            got = {k: state(k, lo, hi) for k in ("master", "m", "v", "working")}
            if w.outer is not None:
                got_outer = dict(master=state("prev", lo, hi), m=state("buf", lo, hi))
            if c + 1 < len(starts):
                nxt = inputs(starts[c + 1], min(w.n, starts[c + 1] + chunk))
            for f in futs:                                   # in index order
                first, ss = f.result()
                seg_acc[:, first:first + ss.shape[1]] += ss
            ref = dict(master=host.master, m=host.m, v=host.v, working=host.working)
            errs = assert_state_parity_fast("%s [%d, %d)" % (w.name, lo, hi), got, ref)
            if w.outer is not None:
                assert_state_parity_fast("%s outer state [%d, %d)" % (w.name, lo, hi), got_outer,
                                         dict(master=host.prev, m=host.buf))
            for k, e in errs.items():
                worst[k] = max(worst.get(k, 0), e)
            del host, got, ref
            if say is not None:
                say("chunk %d/%d: elements [%d, %d) bitwise equal" % (c + 1, len(starts), lo, hi))
    worst["sumsq_rel"] = assert_sumsq(w.name, np.asarray(ss_gpu).reshape(w.A, w.n_seg), seg_acc)
    return worst


def round_cfg(P, w: Workload, step0=None, phase_events=None, dev=None, step_lr=None):
    """The round configuration of workload w (P: the package, kept for the
    callers' signature; see paper_2609_20359_amd.runner)."""
    from paper_2609_20359_amd import runner

    return runner.round_cfg(w, step0=step0, phase_events=phase_events, dev=dev, step_lr=step_lr)


def gpu_round(P, layout, w: Workload, dev: DeviceInputs, seg_sumsq=None, phase_events=None,
              cfg=None):
    """One fl_round (or fl_round_hsdp / fl_round_outer) through the C ABI."""
    from paper_2609_20359_amd import runner

    return runner.gpu_round(layout, w, dev, seg_sumsq=seg_sumsq, phase_events=phase_events,
                            cfg=cfg)


# ---- comparisons -----------------------------------------------------------

def max_rel_err_f32(got, ref):
    """max |got - ref| / max(|ref|, FLT_MIN) over elements where neither is
    NaN; raises if the NaN positions differ."""
    got = np.asarray(got, np.float32)
    ref = np.asarray(ref, np.float32)
    gn, rn = np.isnan(got), np.isnan(ref)
    if not np.array_equal(gn, rn):
        raise AssertionError("NaN positions differ (%d vs %d NaNs)" % (gn.sum(), rn.sum()))
    ok = ~rn
    g, r = got[ok].astype(np.float64), ref[ok].astype(np.float64)
    inf = np.isinf(r) | np.isinf(g)
    if np.any(g[inf] != r[inf]):
        raise AssertionError("infinities differ")
    fin = ~inf
    if not np.any(fin):
        return 0.0
    den = np.maximum(np.abs(r[fin]), np.float64(np.finfo(np.float32).tiny))
    return float(np.max(np.abs(g[fin] - r[fin]) / den))


def _bf16_ordered(u):
    u = np.asarray(u, np.uint16).astype(np.int32)
    return np.where(u & 0x8000, -(u & 0x7FFF), u & 0x7FFF)


def max_bf16_ulp(got, ref):
    """max distance in bf16 ulps (sign-magnitude order); NaN must match NaN."""
    got = np.asarray(got, np.uint16)
    ref = np.asarray(ref, np.uint16)
    gn = ((got & 0x7F80) == 0x7F80) & ((got & 0x7F) != 0)
    rn = ((ref & 0x7F80) == 0x7F80) & ((ref & 0x7F) != 0)
    if not np.array_equal(gn, rn):
        raise AssertionError("bf16 NaN positions differ")
    ok = ~rn
    if not np.any(ok):
        return 0
    return int(np.max(np.abs(_bf16_ordered(got[ok]) - _bf16_ordered(ref[ok]))))


def assert_state_parity(tag, gpu, ref, bitwise=False):
    """gpu/ref: dicts with master, m, v (f32) and working (u16).  bitwise:
    every element bitwise equal, except that NaNs need only match in
    position (x86 and gfx950 make different default NaNs)."""
    errs = {}
    for k in ("master", "m", "v"):
        if k not in ref:
            continue
        e = max_rel_err_f32(gpu[k], ref[k])
        errs[k] = e
        assert e <= TOL_F32_REL, "%s: %s max rel err %.3g > %g" % (tag, k, e, TOL_F32_REL)
        if bitwise:
            g32, r32 = np.asarray(gpu[k], np.float32), np.asarray(ref[k], np.float32)
            ok = ~np.isnan(r32)
            assert np.array_equal(g32[ok].view(np.uint32), r32[ok].view(np.uint32)), \
                "%s: %s not bitwise" % (tag, k)
    if "working" in ref:
        u = max_bf16_ulp(gpu["working"], ref["working"])
        errs["working_ulp"] = u
        assert u <= TOL_BF16_ULP, "%s: working %d bf16 ulp > %d" % (tag, u, TOL_BF16_ULP)
        if bitwise:
            gw, rw = np.asarray(gpu["working"], np.uint16), np.asarray(ref["working"], np.uint16)
            ok = ~(((rw & 0x7F80) == 0x7F80) & ((rw & 0x7F) != 0))
            assert np.array_equal(gw[ok], rw[ok]), "%s: working not bitwise" % tag
    return errs


def assert_sumsq(tag, got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    nan_g, nan_r = np.isnan(got), np.isnan(ref)
    assert np.array_equal(nan_g, nan_r), "%s: sumsq NaN positions" % tag
    inf_g, inf_r = np.isinf(got), np.isinf(ref)
    assert np.array_equal(inf_g, inf_r) and np.array_equal(got[inf_r], ref[inf_r]), \
        "%s: sumsq infinities" % tag
    ok = ~nan_r & ~inf_r
    rel = np.abs(got[ok] - ref[ok]) / np.maximum(np.abs(ref[ok]), 1e-300)
    worst = float(rel.max()) if rel.size else 0.0
    assert worst <= TOL_SUMSQ_REL, "%s: seg_sumsq rel err %.3g" % (tag, worst)
    return worst
