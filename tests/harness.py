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
    """Run the oracle round (FL+FSDP, or FL+HSDP when w.H > 1) in place on host
    arrays.  Returns the per-step per-segment sums of squares or None.
    clip_totals: per-step whole-shard sums of squares to clip against when the
    host arrays hold only a sample of the shard."""
    seg_off = w.seg_offsets if seg_off is None else seg_off
    seg_decay = w.seg_decay if seg_decay is None else seg_decay
    if w.outer is not None:
        return orc.round_outer(seg_off, seg_decay, w.R, w.G, w.A, w.self_group, w.grad_scale,
                               w.hp, w.step0, w.weights, w.outer, host.grads, host.replicas,
                               host.prev, host.buf, host.master, host.m, host.v, host.working,
                               want_sumsq=want_sumsq, max_grad_norm=w.max_grad_norm,
                               clip_totals=clip_totals, step_lr=step_lr)
    if w.H > 1:
        return orc.round_hsdp(seg_off, seg_decay, w.R, w.H, w.replica, 1.0 / w.H, w.hsdp_member,
                              w.G, w.A, w.self_group, w.grad_scale, w.hp, w.step0, w.weights,
                              host.grads, host.replica_wires, host.replicas, host.bcast,
                              host.master, host.m, host.v, host.working, want_sumsq=want_sumsq,
                              max_grad_norm=w.max_grad_norm, clip_totals=clip_totals,
                              step_lr=step_lr)
    return orc.round(seg_off, seg_decay, w.R, w.G, w.A, w.self_group, w.grad_scale, w.hp,
                     w.step0, w.weights, host.grads, host.replicas, host.master, host.m, host.v,
                     host.working, want_sumsq=want_sumsq, max_grad_norm=w.max_grad_norm,
                     clip_totals=clip_totals, step_lr=step_lr)


def clip_totals(orc, w: Workload, chunk=1 << 24, say=None):
    """Whole-shard sum of squares of each local step's reduced gradient, in
    index order, one chunk of host-regenerated peer gradients at a time (for a
    clipped round whose oracle sees only a sample of the shard)."""
    assert w.H == 1, "the FL+HSDP clip norm is that of the replica average"
    steps = [tuple(w.grad_index[a * w.R:(a + 1) * w.R]) for a in range(w.A)]
    done = {}
    for key in dict.fromkeys(steps):
        acc = 0.0
        for c, lo in enumerate(range(0, w.n, chunk)):
            k = min(chunk, w.n - lo)
            acc = orc.grad_total([host_fill(w.grad_specs[j], lo, k) for j in key],
                                 w.grad_scale, acc)
            if say is not None and c % 16 == 15:
                say("clip total: %d of %d elements" % (lo + k, w.n))
        done[key] = acc
    return [done[key] for key in steps]


def round_cfg(P, w: Workload, step0=None, phase_events=None, dev=None, step_lr=None):
    """The round configuration of workload w (with dev: its gradient scratch,
    if the workload has one)."""
    scratch = None if dev is None else getattr(dev, "grad_scratch", None)
    return P.make_round_cfg(w.R, w.G, w.A, w.weights, w.hp, self_group=w.self_group,
                            grad_scale=w.grad_scale, step0=w.step0 if step0 is None else step0,
                            phase_events=phase_events, max_grad_norm=w.max_grad_norm,
                            grad_scratch=scratch, step_lr=step_lr)


def gpu_round(P, layout, w: Workload, dev: DeviceInputs, seg_sumsq=None, phase_events=None,
              cfg=None):
    """One fl_round (or fl_round_hsdp when w.H > 1) through the C ABI."""
    if cfg is None:
        cfg = round_cfg(P, w, phase_events=phase_events, dev=dev)
    if w.outer is not None:
        P.fl_round_outer(layout, cfg, w.outer, dev.grads, dev.replicas, dev.prev, dev.buf,
                         dev.master, dev.m, dev.v, dev.working, seg_sumsq=seg_sumsq)
    elif w.H > 1:
        hc = P.make_hsdp_cfg(w.H, w.replica, 1.0 / w.H, w.hsdp_member)
        P.fl_round_hsdp(layout, cfg, hc, dev.grads, dev.replica_wires, dev.wire,
                        dev.replicas if w.hsdp_member else None,
                        None if w.hsdp_member else dev.bcast, dev.master, dev.m, dev.v,
                        dev.working, seg_sumsq=seg_sumsq)
    else:
        P.fl_round(layout, cfg, dev.grads, dev.replicas, dev.master, dev.m, dev.v, dev.working,
                   seg_sumsq=seg_sumsq)
    return cfg


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
