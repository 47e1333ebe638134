"""Pins of the CPU oracle to things other than itself.

Each pin_* function takes an ``oracle.Oracle`` and raises AssertionError when
the oracle disagrees with an independent reference: torch's own bf16 cast,
torch.optim.AdamW run in float64, float64 numpy sums, closed forms of the
method's special cases, hand-derived exact cases (tests/golden), and a
straight-line float64 recomputation of whole rounds with propagated
rounding-error bounds.  test_oracle_pins.py runs them on the oracle;
test_oracle_mutants.py runs them on copies of the oracle with planted
mistakes and requires that every mistake is caught.
"""
import json
import os

import numpy as np
import torch

U = 2.0 ** -24          # unit roundoff of binary32
TINY = 2.0 ** -149      # smallest subnormal binary32

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

STD_HP = dict(lr=3e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)
# Exaggerated hyperparameters: make every term of the update large enough that
# dropping or misplacing it moves the result far outside rounding error.
BIG_HP = dict(lr=0.05, beta1=0.8, beta2=0.9, eps=1e-3, weight_decay=0.5)


# ---- independent helpers (no oracle code) --------------------------------

def bf16_decode(u16):
    """bf16 bits -> float64 values, by numpy bit manipulation."""
    u = np.asarray(u16, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def torch_bf16_bits(f32):
    """float32 -> bf16 bits via torch's own conversion."""
    t = torch.from_numpy(np.ascontiguousarray(f32, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def f32(x):
    return np.float32(x)


def rng(seed):
    return np.random.default_rng(seed)


def random_bf16(r, n, std=1e-3):
    return torch_bf16_bits((r.standard_normal(n) * std).astype(np.float32))


def bf16_boundary_between(lo, hi):
    """True where the closed interval [lo, hi] (float64) contains a bf16
    rounding boundary, i.e. where the bf16 rounding of a value in it is not
    unique."""
    lo32 = lo.astype(np.float32)
    hi32 = hi.astype(np.float32)
    a = torch_bf16_bits(np.nextafter(lo32, np.float32(-np.inf)))
    b = torch_bf16_bits(np.nextafter(hi32, np.float32(np.inf)))
    return a != b


def _hp_f(hp):
    return {k: float(np.float32(v)) for k, v in hp.items()}


# ---- bf16 conversions ------------------------------------------------------

def pin_bf16_decode_all_patterns(orc):
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ours = orc.bf16_to_f32(bits).view(np.uint32)
    ref = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(torch.float32)
    ref = ref.numpy().view(np.uint32)
    assert np.array_equal(ours, ref), "bf16 -> f32 differs from torch"


def _conversion_cases(seed=0):
    r = rng(seed)
    vals = [r.standard_normal(20000) * 10.0 ** r.integers(-40, 38, 20000)]
    # ties: lower 16 bits exactly 0x8000, with even and odd upper halves
    up = r.integers(0, 0x7F7F, 4000, dtype=np.uint32)
    ties = ((up << 16) | 0x8000).astype(np.uint32)
    near = np.concatenate([ties - 1, ties + 1, ties, ties | 0x80000000])
    vals.append(near.view(np.float32))
    special = np.array([0x00000000, 0x80000000, 0x7F800000, 0xFF800000, 0x7F7FFFFF, 0xFF7FFFFF,
                        0x7F7F8000, 0x7F7F7FFF, 0x00800000, 0x00000001, 0x00008000, 0x00018000,
                        0x007FFFFF, 0x80008000, 0x3F808000, 0x3F818000, 0x3F80FFFF],
                       dtype=np.uint32).view(np.float32)
    vals.append(special)
    return np.concatenate([v.astype(np.float32) for v in vals])


def pin_bf16_encode_matches_torch(orc):
    x = _conversion_cases()
    ours = orc.f32_to_bf16(x)
    ref = torch_bf16_bits(x)
    bad = np.nonzero(ours != ref)[0]
    assert bad.size == 0, "f32 -> bf16 differs from torch at %d values, e.g. %s -> %04x vs %04x" % (
        bad.size, hex(x[bad[0]:bad[0] + 1].view(np.uint32)[0]), ours[bad[0]], ref[bad[0]])


def pin_bf16_encode_nan(orc):
    nans = np.array([0x7FC00000, 0xFFC00000, 0x7F800001, 0xFF800001, 0x7FBFFFFF, 0x7F80FFFF,
                     0x7F810000], dtype=np.uint32).view(np.float32)
    out = orc.f32_to_bf16(nans)
    dec = bf16_decode(out)
    assert np.all(np.isnan(dec)), "a NaN did not stay NaN"
    assert np.array_equal(out >> 15, (nans.view(np.uint32) >> 31).astype(np.uint16)), "NaN sign lost"
    assert np.all(out & 0x0040), "NaN not quiet"


# ---- (a1) peer reduction ---------------------------------------------------

def pin_reduce_vs_float64_sum(orc):
    r = rng(1)
    for R, scale in ((1, 1.0), (3, 1.0 / 3.0), (8, 0.125), (16, 1.0 / 16), (5, 0.7)):
        n = 4096
        grads = [random_bf16(r, n, std=10.0 ** r.uniform(-5, 1)) for _ in range(R)]
        g = orc.shard_reduce(grads, scale).astype(np.float64)
        dec = np.stack([bf16_decode(x) for x in grads])
        s = float(np.float32(scale))
        exact = dec.sum(0) * s
        bound = (R + 1) * U * np.abs(dec).sum(0) * abs(s) + TINY
        err = np.abs(g - exact)
        assert np.all(err <= bound), "reduce R=%d off by %g (bound %g)" % (
            R, err.max(), bound[np.argmax(err - bound)])


def pin_reduce_identical_peers_exact(orc):
    r = rng(2)
    x = random_bf16(r, 3000, std=0.5)
    for R in (1, 2, 4, 8, 16):
        g = orc.shard_reduce([x] * R, 1.0 / R)
        assert np.array_equal(g.astype(np.float64), bf16_decode(x)), "mean of %d equal peers" % R


# ---- (a5) per-segment sum of squares ----------------------------------------

def pin_seg_sumsq_vs_numpy(orc):
    r = rng(3)
    sizes = r.integers(1, 400, 40)
    off = np.zeros(sizes.size + 1, np.int64)
    off[1:] = np.cumsum(sizes)
    g = (r.standard_normal(off[-1]) * 1e-3).astype(np.float32)
    ss = orc.seg_sumsq(off, g)
    g64 = g.astype(np.float64)
    ref = np.array([np.sum(g64[off[s]:off[s + 1]] ** 2) for s in range(sizes.size)])
    assert np.allclose(ss, ref, rtol=1e-12, atol=0), "per-segment sum of squares"


# ---- (a2) AdamW --------------------------------------------------------------

def _torch_adamw_run(hp, p0, grads_per_step, decay_mask):
    """torch.optim.AdamW in float64 (single-tensor path): one param group with
    weight decay for decay_mask elements, one without."""
    hpf = _hp_f(hp)
    p_dec = torch.tensor(p0[decay_mask], dtype=torch.float64, requires_grad=True)
    p_nod = torch.tensor(p0[~decay_mask], dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW(
        [dict(params=[p_dec], weight_decay=hpf["weight_decay"]),
         dict(params=[p_nod], weight_decay=0.0)],
        lr=hpf["lr"], betas=(hpf["beta1"], hpf["beta2"]), eps=hpf["eps"], foreach=False,
        fused=False, amsgrad=False, maximize=False)
    hist = []
    for g in grads_per_step:
        p_dec.grad = torch.tensor(g[decay_mask], dtype=torch.float64)
        p_nod.grad = torch.tensor(g[~decay_mask], dtype=torch.float64)
        opt.step()
        out = {}
        for key, src in (("p", lambda t: t.detach()), ("m", lambda t: opt.state[t]["exp_avg"]),
                         ("v", lambda t: opt.state[t]["exp_avg_sq"])):
            a = np.empty(p0.size)
            a[decay_mask] = src(p_dec).numpy()
            a[~decay_mask] = src(p_nod).numpy()
            out[key] = a
        hist.append(out)
    return hist


def _adamw_bounds(hp, t_max, p0, grads_per_step, decay_mask):
    """Propagated worst-case bounds on |fp32 oracle - exact| for p, m, v."""
    h = _hp_f(hp)
    b1, b2, lr, wd, eps = h["beta1"], h["beta2"], h["lr"], h["weight_decay"], h["eps"]
    p = p0.astype(np.float64).copy()
    m = np.zeros_like(p)
    v = np.zeros_like(p)
    ep = np.zeros_like(p)
    em = np.zeros_like(p)
    ev = np.zeros_like(p)
    mabs = np.zeros_like(p)
    decay = np.where(decay_mask, 1.0 - lr * wd, 1.0)
    out = []
    for t, g in enumerate(grads_per_step, start=1):
        g = g.astype(np.float64)
        mabs = b1 * mabs + (1 - b1) * np.abs(g)
        m = b1 * m + (1 - b1) * g
        em = b1 * em + 4 * U * mabs
        v = b2 * v + (1 - b2) * g * g
        ev = b2 * ev + 5 * U * v
        bc1 = 1 - b1 ** t
        bc2s = np.sqrt(1 - b2 ** t)
        s = np.sqrt(v)
        es = np.minimum(ev / np.maximum(2 * s, TINY), np.sqrt(ev)) + U * s
        den = s / bc2s + eps
        eden = es / bc2s + 3 * U * s / bc2s + U * den
        ratio = m / den
        eratio = em / den + mabs / den * (eden / den) + 2 * U * mabs / den
        step = lr / bc1
        upd = step * ratio
        eupd = step * eratio + 3 * U * step * mabs / den
        pd = p * decay
        ep = decay * ep + 2 * U * np.abs(pd)
        p = pd - upd
        ep = ep + eupd + U * np.abs(p)
        out.append(dict(p=(p, 2 * ep + TINY), m=(m, 2 * em + TINY), v=(v, 2 * ev + TINY)))
    return out


def _check_close(name, got, ref, bound):
    err = np.abs(got.astype(np.float64) - ref)
    bad = np.nonzero(~(err <= bound))[0]
    assert bad.size == 0, "%s: %d elements out of bound, worst |err| %g at ref %g (bound %g)" % (
        name, bad.size, err[bad].max(), ref[bad[np.argmax(err[bad])]],
        bound[bad[np.argmax(err[bad])]])


def pin_adamw_vs_torch_float64(orc):
    r = rng(4)
    for hp in (STD_HP, BIG_HP):
        n = 2048
        p0 = (r.standard_normal(n) * 0.02).astype(np.float32)
        mask = np.zeros(n, bool)
        mask[:1500] = True   # first segment decays, second does not
        off = np.array([0, 1500, n], np.int64)
        flags = np.array([1, 0], np.uint8)
        steps = 5
        gs = [(r.standard_normal(n) * 10.0 ** r.uniform(-4, -1)).astype(np.float32)
              for _ in range(steps)]
        gs[2][::7] = 0.0
        ref = _torch_adamw_run(hp, p0, gs, mask)
        bounds = _adamw_bounds(hp, steps, p0, gs, mask)
        master = p0.copy()
        m = np.zeros(n, np.float32)
        v = np.zeros(n, np.float32)
        for t in range(1, steps + 1):
            orc.adamw_step(off, flags, hp, t, gs[t - 1], master, m, v)
            for key, arr in (("p", master), ("m", m), ("v", v)):
                _, bnd = bounds[t - 1][key]
                _check_close("adamw %s t=%d lr=%g" % (key, t, hp["lr"]), arr, ref[t - 1][key], bnd)


def pin_adamw_first_step_closed_form(orc):
    """t = 1 from m = v = 0: p1 = p0 (1 - lr wd) - lr g / (|g| + eps),
    m1 = (1 - b1) g, v1 = (1 - b2) g^2."""
    r = rng(5)
    for hp in (STD_HP, BIG_HP):
        h = _hp_f(hp)
        n = 4096
        p0 = (r.standard_normal(n) * 0.02).astype(np.float32)
        g = (r.standard_normal(n) * 1e-3).astype(np.float32)
        master, m, v = p0.copy(), np.zeros(n, np.float32), np.zeros(n, np.float32)
        work = np.zeros(n, np.uint16)
        orc.adamw_step(np.array([0, n], np.int64), np.array([1], np.uint8), hp, 1, g, master, m,
                       v, work)
        p64, g64 = p0.astype(np.float64), g.astype(np.float64)
        want = p64 * (1 - h["lr"] * h["weight_decay"]) - h["lr"] * g64 / (np.abs(g64) + h["eps"])
        bound = 16 * U * (np.abs(p64) + h["lr"]) + TINY
        _check_close("first-step p", master, want, bound)
        _check_close("first-step m", m, (1 - h["beta1"]) * g64, 2 * U * np.abs(g64) + TINY)
        _check_close("first-step v", v, (1 - h["beta2"]) * g64 * g64, 3 * U * g64 * g64 + TINY)
        assert np.array_equal(work, torch_bf16_bits(master)), "working copy is not bf16(master)"


def pin_adamw_zero_grad(orc):
    """g = 0 at t = 1: m = v = 0 and p = p0 * decay exactly."""
    r = rng(6)
    n = 1000
    p0 = (r.standard_normal(n) * 0.02).astype(np.float32)
    for hp in (STD_HP, BIG_HP):
        h = _hp_f(hp)
        off = np.array([0, 600, n], np.int64)
        flags = np.array([1, 0], np.uint8)
        master, m, v = p0.copy(), np.zeros(n, np.float32), np.zeros(n, np.float32)
        orc.adamw_step(off, flags, hp, 1, np.zeros(n, np.float32), master, m, v)
        decay = np.float32(1.0 - h["lr"] * h["weight_decay"])
        assert np.array_equal(master[:600], p0[:600] * decay), "zero grad, decayed segment"
        assert np.array_equal(master[600:], p0[600:]), "zero grad, undecayed segment"
        assert not m.any() and not v.any(), "zero grad moved m or v"


def pin_adamw_lr_zero(orc):
    r = rng(7)
    n = 1000
    p0 = (r.standard_normal(n) * 0.02).astype(np.float32)
    hp = dict(BIG_HP, lr=0.0)
    master, m, v = p0.copy(), np.zeros(n, np.float32), np.zeros(n, np.float32)
    g = (r.standard_normal(n) * 1e-2).astype(np.float32)
    for t in (1, 2, 3):
        orc.adamw_step(np.array([0, n], np.int64), np.array([1], np.uint8), hp, t, g, master, m, v)
    assert np.array_equal(master, p0), "lr = 0 changed the master weights"
    assert m.any() and v.any(), "lr = 0 must still update the moments"


# ---- (a3) FedAvg -------------------------------------------------------------

def pin_fedavg_identical_replicas(orc):
    r = rng(8)
    x = random_bf16(r, 5000, std=0.02)
    for G in (1, 2, 3, 4, 7, 8, 16):
        w = r.uniform(0.1, 5.0, G).astype(np.float32)
        master, work = orc.fedavg([x] * G, w)
        assert np.array_equal(work, x), "FedAvg of identical replicas changed them (G=%d)" % G
        err = np.abs(master.astype(np.float64) - bf16_decode(x))
        assert np.all(err <= (G + 2) * U * np.abs(bf16_decode(x)) + TINY), "identity G=%d" % G
        if G & (G - 1) == 0:
            master, _ = orc.fedavg([x] * G, np.ones(G, np.float32))
            assert np.array_equal(master.astype(np.float64), bf16_decode(x)), "equal weights G=%d" % G


def pin_fedavg_two_group_mean(orc):
    r = rng(9)
    x0, x1 = random_bf16(r, 5000, 0.02), random_bf16(r, 5000, 0.02)
    master, work = orc.fedavg([x0, x1], np.array([0.5, 0.5], np.float32))
    want = ((bf16_decode(x0) + bf16_decode(x1)) / 2).astype(np.float32)
    assert np.array_equal(master, want), "two-group mean is not the arithmetic mean"
    assert np.array_equal(work, torch_bf16_bits(want)), "working copy of the mean"


def pin_fedavg_vs_float64_average(orc):
    r = rng(10)
    for G in (2, 3, 8, 16):
        n = 4096
        reps = [random_bf16(r, n, 0.02) for _ in range(G)]
        w = r.integers(1, 17, G).astype(np.float32)
        master, work = orc.fedavg(reps, w)
        dec = np.stack([bf16_decode(x) for x in reps])
        wn = w.astype(np.float64) / w.astype(np.float64).sum()
        exact = (wn[:, None] * dec).sum(0)
        bound = (G + 2) * U * (wn[:, None] * np.abs(dec)).sum(0) + TINY
        _check_close("fedavg G=%d" % G, master, exact, bound)
        uniq = ~bf16_boundary_between(exact - bound, exact + bound)
        assert np.array_equal(work[uniq], torch_bf16_bits(exact.astype(np.float32))[uniq]), \
            "FedAvg working copy G=%d" % G


def pin_fedavg_weight_scale_invariance(orc):
    """A weighted average depends on the weights only up to a common factor."""
    r = rng(11)
    reps = [random_bf16(r, 3000, 0.02) for _ in range(6)]
    w = r.integers(1, 17, 6).astype(np.float32)
    a, _ = orc.fedavg(reps, w)
    b, _ = orc.fedavg(reps, w * np.float32(4.0))
    assert np.array_equal(a, b), "weights w and 4w give different averages"


# ---- hand-derived exact cases (tests/golden/hand_cases.json) ----------------

def pin_golden_hand_cases(orc):
    with open(os.path.join(GOLDEN, "hand_cases.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        kind = c["op"]
        if kind == "reduce":
            grads = [torch_bf16_bits(np.array(x, np.float32)) for x in c["peers"]]
            g = orc.shard_reduce(grads, c["grad_scale"])
            assert np.array_equal(g, np.array(c["expect_g"], np.float32)), c["name"]
        elif kind == "fedavg":
            reps = [torch_bf16_bits(np.array(x, np.float32)) for x in c["replicas"]]
            master, work = orc.fedavg(reps, np.array(c["weights"], np.float32))
            assert np.array_equal(master, np.array(c["expect_master"], np.float32)), c["name"]
            assert np.array_equal(work, torch_bf16_bits(np.array(c["expect_master"], np.float32))), c["name"]
        elif kind == "adamw":
            n = len(c["p0"])
            master = np.array(c["p0"], np.float32)
            m = np.array(c["m0"], np.float32)
            v = np.array(c["v0"], np.float32)
            orc.adamw_step(np.array([0, n], np.int64), np.array([c["decay"]], np.uint8), c["hp"],
                           c["t"], np.array(c["g"], np.float32), master, m, v)
            assert np.array_equal(master, np.array(c["expect_p"], np.float32)), c["name"]
            assert np.array_equal(m, np.array(c["expect_m"], np.float32)), c["name"]
            assert np.array_equal(v, np.array(c["expect_v"], np.float32)), c["name"]
        else:
            raise AssertionError("unknown golden op " + kind)


# ---- (a4) whole rounds: float64 brute force with error bounds ---------------

def _bf_steps(hp, seg_off, seg_decay, step0, gsteps, p0, m0, v0, lrs=None):
    """float64 AdamW over the given per-step (g, bound on |fp32 g - g|) with
    propagated bounds on the distance of the binary32 evaluation; lrs: one
    learning rate per step (else hp's)."""
    h = _hp_f(hp)
    b1, b2, lr, wd, eps = h["beta1"], h["beta2"], h["lr"], h["weight_decay"], h["eps"]
    n = int(seg_off[-1])
    decay_flag = np.zeros(n, bool)
    for s in range(len(seg_off) - 1):
        decay_flag[seg_off[s]:seg_off[s + 1]] = bool(seg_decay[s])
    p = p0.astype(np.float64).copy()
    m = m0.astype(np.float64).copy()
    v = v0.astype(np.float64).copy()
    ep = np.zeros(n)
    em = np.zeros(n)
    ev = np.zeros(n)
    mabs = np.abs(m)
    for a, (g, eg) in enumerate(gsteps):
        t = step0 + a
        if lrs is not None:
            lr = float(np.float32(lrs[a]))
        decay = np.where(decay_flag, 1.0 - lr * wd, 1.0)
        gab = np.abs(g) + eg
        mabs = b1 * mabs + (1 - b1) * gab
        m = b1 * m + (1 - b1) * g
        em = b1 * em + (1 - b1) * eg + 4 * U * mabs
        v = b2 * v + (1 - b2) * g * g
        ev = b2 * ev + (1 - b2) * (2 * np.abs(g) * eg + eg * eg) + 5 * U * (b2 * v + (1 - b2) * gab * gab)
        bc1 = 1 - b1 ** t
        bc2s = np.sqrt(1 - b2 ** t)
        s = np.sqrt(v)
        es = np.minimum(ev / np.maximum(2 * s, TINY), np.sqrt(ev)) + U * s
        den = s / bc2s + eps
        eden = es / bc2s + 3 * U * (s + es) / bc2s + U * den
        dlow = np.maximum(den - eden, eps * 0.5)
        ratio = m / den
        eratio = em / dlow + mabs * eden / (dlow * dlow) + 2 * U * mabs / dlow
        step = lr / bc1
        upd = step * ratio
        eupd = step * eratio + 3 * U * step * mabs / dlow
        pd = p * decay
        ep = decay * ep + 2 * U * (np.abs(pd) + ep)
        p = pd - upd
        ep = ep + eupd + U * (np.abs(p) + ep)
    return (p, 2 * ep + TINY), (m, 2 * em + TINY), (v, 2 * ev + TINY)


def _bf_reduce(grads, scale):
    """float64 value of an ascending fp32 sum of bf16 arrays times scale, with
    a bound on the binary32 evaluation's distance."""
    dec = np.stack([bf16_decode(x) for x in grads])
    s_scale = float(np.float32(scale))
    return dec.sum(0) * s_scale, (len(grads) + 1) * U * np.abs(dec).sum(0) * abs(s_scale)


def _bf_fedavg(weights, reps):
    wv = np.asarray(weights, np.float32).astype(np.float64)
    wn = wv / wv.sum()
    dec = np.stack([bf16_decode(x) for x in reps])
    xbar = (wn[:, None] * dec).sum(0)
    return xbar, 2 * (len(reps) + 2) * U * (wn[:, None] * np.abs(dec)).sum(0) + TINY


def _resolve_bf16(val, bnd, oracle_bits):
    """bf16 rounding of a value known within +-bnd: unique where no rounding
    boundary lies in the interval (then it must equal oracle_bits if given);
    elsewhere the oracle's bits are taken after checking that they are the
    rounding of some value in the interval.  Returns (bits, ambiguous mask)."""
    amb = bf16_boundary_between(val - bnd, val + bnd)
    ref = torch_bf16_bits(val.astype(np.float32))
    if oracle_bits is None:
        return ref, amb
    lo = bf16_decode(torch_bf16_bits(np.nextafter((val - bnd).astype(np.float32), np.float32(-np.inf))))
    hi = bf16_decode(torch_bf16_bits(np.nextafter((val + bnd).astype(np.float32), np.float32(np.inf))))
    got = bf16_decode(oracle_bits)
    ok = (~amb & (oracle_bits == ref)) | (amb & (got >= lo) & (got <= hi))
    assert np.all(ok), "bf16 rounding outside the candidates"
    return np.where(amb, oracle_bits, ref), amb


def brute_force_round(hp, seg_off, seg_decay, R, G, A, self_group, grad_scale, step0, weights,
                      grads, replicas, p0, m0, v0, oracle_working_after_steps=None):
    """Straight-line float64 recomputation of one round, with a propagated
    bound on the distance of any binary32 evaluation in the fixed order from
    the exact result.  Returns dict of (value, bound) plus the per-step g and
    its bound, and the masks of elements whose bf16 rounding is ambiguous."""
    gsteps = [_bf_reduce(grads[a * R:(a + 1) * R], grad_scale) for a in range(A)]
    (p, ep), (m, em), (v, ev) = _bf_steps(hp, seg_off, seg_decay, step0, gsteps, p0, m0, v0)
    amb_w = bf16_boundary_between(p - ep, p + ep)
    w_ref = torch_bf16_bits(p.astype(np.float32))
    if oracle_working_after_steps is not None:
        w_own = np.where(amb_w, oracle_working_after_steps, w_ref)
    else:
        w_own = w_ref
    reps = [w_own if k == self_group else replicas[k] for k in range(G)]
    xbar, ex = _bf_fedavg(weights, reps)
    amb_f = bf16_boundary_between(xbar - ex, xbar + ex)
    return dict(master=(xbar, ex), m=(m, em), v=(v, ev), p_steps=(p, ep), w_own=w_own,
                amb_own=amb_w, amb_final=amb_f, g=gsteps)


def _random_round_case(r, R, G, A, n=16, hp=None):
    cuts = np.sort(r.choice(np.arange(1, n), size=r.integers(0, 4), replace=False))
    off = np.concatenate([[0], cuts, [n]]).astype(np.int64)
    flags = r.integers(0, 2, off.size - 1).astype(np.uint8)
    grads = [random_bf16(r, n, std=10.0 ** r.uniform(-4, -1)) for _ in range(A * R)]
    p0 = (r.standard_normal(n) * 0.02).astype(np.float32)
    reps = [None if k == 0 else torch_bf16_bits((p0 + r.standard_normal(n) * 1e-3).astype(np.float32))
            for k in range(G)]
    self_group = int(r.integers(0, G))
    if self_group != 0:
        reps[0], reps[self_group] = reps[self_group], None
    w = r.uniform(0.1, 2.0, G).astype(np.float32)
    m0 = (r.standard_normal(n) * 1e-4).astype(np.float32)
    v0 = (np.abs(r.standard_normal(n)) * 1e-7).astype(np.float32)
    return dict(seg_off=off, seg_decay=flags, R=R, G=G, A=A, self_group=self_group,
                grad_scale=1.0 / R, step0=int(r.integers(1, 20)), weights=w, grads=grads,
                replicas=reps, p0=p0, m0=m0, v0=v0)


def check_round_against_brute_force(orc, hp, case):
    c = case
    master, m, v = c["p0"].copy(), c["m0"].copy(), c["v0"].copy()
    work = torch_bf16_bits(master)
    # the oracle's own working copy after the local steps (used only where the
    # bf16 rounding of the float64 value is ambiguous)
    mw, mm, mv = master.copy(), m.copy(), v.copy()
    ww = work.copy()
    for a in range(c["A"]):
        g = orc.shard_reduce(c["grads"][a * c["R"]:(a + 1) * c["R"]], c["grad_scale"])
        orc.adamw_step(c["seg_off"], c["seg_decay"], hp, c["step0"] + a, g, mw, mm, mv, ww)
    ss = orc.round(c["seg_off"], c["seg_decay"], c["R"], c["G"], c["A"], c["self_group"],
                   c["grad_scale"], hp, c["step0"], c["weights"], c["grads"], c["replicas"],
                   master, m, v, work, want_sumsq=True)
    bf = brute_force_round(hp, c["seg_off"], c["seg_decay"], c["R"], c["G"], c["A"],
                           c["self_group"], c["grad_scale"], c["step0"], c["weights"], c["grads"],
                           c["replicas"], c["p0"], c["m0"], c["v0"], oracle_working_after_steps=ww)
    tag = "R=%d G=%d A=%d self=%d" % (c["R"], c["G"], c["A"], c["self_group"])
    own_ok = bf["amb_own"] | (ww == bf["w_own"])
    assert np.all(own_ok), "working copy after the local steps, " + tag
    for key, arr in (("master", master), ("m", m), ("v", v)):
        val, bnd = bf[key]
        _check_close("round %s %s" % (key, tag), arr, val, bnd)
    xbar, _ = bf["master"]
    uniq = ~bf["amb_final"]
    assert np.array_equal(work[uniq], torch_bf16_bits(xbar.astype(np.float32))[uniq]), \
        "round working copy " + tag
    assert np.array_equal(work, torch_bf16_bits(master)), "working != bf16(master) " + tag
    off = c["seg_off"]
    for a, (g, eg) in enumerate(bf["g"]):
        for s in range(off.size - 1):
            sl = slice(off[s], off[s + 1])
            want = np.sum(g[sl] ** 2)
            bound = np.sum(2 * np.abs(g[sl]) * eg[sl] + eg[sl] ** 2) * 2 + 1e-12 * want + TINY
            assert abs(ss[a, s] - want) <= bound, "seg_sumsq step %d seg %d %s" % (a, s, tag)


def pin_round_brute_force_16(orc):
    """Every (R, G, A) in {1..4}^3 on 16-element shards with random segment
    splits, decay flags, self group, weights and starting state."""
    r = rng(12)
    for hp in (STD_HP, BIG_HP):
        for R in range(1, 5):
            for G in range(1, 5):
                for A in range(1, 5):
                    check_round_against_brute_force(orc, hp, _random_round_case(r, R, G, A))


def pin_round_single_step_single_group(orc):
    """A = 1, G = 1, w = 1: one AdamW step, then FedAvg is the identity on the
    working copy, so master becomes the widened working copy."""
    r = rng(13)
    n = 777
    c = _random_round_case(r, 2, 1, 1, n=n)
    c["self_group"] = 0
    c["replicas"] = [None]
    c["weights"] = np.array([1.0], np.float32)
    master, m, v = c["p0"].copy(), c["m0"].copy(), c["v0"].copy()
    work = np.zeros(n, np.uint16)
    orc.round(c["seg_off"], c["seg_decay"], 2, 1, 1, 0, 0.5, STD_HP, c["step0"], c["weights"],
              c["grads"], c["replicas"], master, m, v, work)
    bf = brute_force_round(STD_HP, c["seg_off"], c["seg_decay"], 2, 1, 1, 0, 0.5, c["step0"],
                           c["weights"], c["grads"], c["replicas"], c["p0"], c["m0"], c["v0"])
    p, ep = bf["p_steps"]
    uniq = ~bf["amb_own"]
    assert np.array_equal(work[uniq], torch_bf16_bits(p.astype(np.float32))[uniq]), "A=1,G=1 working"
    assert np.array_equal(master.astype(np.float64), bf16_decode(work)), "A=1,G=1 master"


def pin_round_uses_own_working_copy(orc):
    """The own replica entering FedAvg is this group's freshly updated bf16
    working copy: with G = 2 and the other replica equal to the pre-round
    working copy, a round with lr > 0 must differ from the stale average."""
    r = rng(14)
    n = 512
    c = _random_round_case(r, 1, 2, 2, n=n)
    c["self_group"] = 1
    stale = torch_bf16_bits(c["p0"])
    c["replicas"] = [stale, None]
    c["weights"] = np.array([0.0, 1.0], np.float32)
    master, m, v = c["p0"].copy(), c["m0"].copy(), c["v0"].copy()
    work = stale.copy()
    orc.round(c["seg_off"], c["seg_decay"], 1, 2, 2, 1, 1.0, BIG_HP, c["step0"], c["weights"],
              c["grads"], c["replicas"], master, m, v, work)
    # weight 0 on the other group: the result is the own updated copy
    bf = brute_force_round(BIG_HP, c["seg_off"], c["seg_decay"], 1, 2, 2, 1, 1.0, c["step0"],
                           c["weights"], c["grads"], c["replicas"], c["p0"], c["m0"], c["v0"])
    xbar, ex = bf["master"]
    _check_close("own copy", master, xbar, ex)
    assert not np.array_equal(work, stale), "round did not use the updated working copy"


# ---- FL+HSDP: two-tier gradient average and broadcast receive -------------

def pin_reduce_wire_vs_float64(orc):
    r = rng(15)
    for R, scale in ((1, 1.0), (4, 0.25), (8, 0.125), (5, 0.2)):
        grads = [random_bf16(r, 6000, std=10.0 ** r.uniform(-4, 0)) for _ in range(R)]
        wire = orc.shard_reduce_wire(grads, scale)
        val, bnd = _bf_reduce(grads, scale)
        _resolve_bf16(val, bnd + TINY, wire)


def pin_broadcast_recv(orc):
    r = rng(16)
    recv = (r.standard_normal(3000) * 0.02).astype(np.float32)
    recv[:5] = [0.0, -0.0, np.inf, 3e38, 1e-40]
    master = np.zeros(3000, np.float32)
    work = np.zeros(3000, np.uint16)
    orc.broadcast_recv(recv, master, work)
    assert np.array_equal(master.view(np.uint32), recv.view(np.uint32)), "master != received"
    assert np.array_equal(work, torch_bf16_bits(recv)), "working != bf16(received)"


def _random_hsdp_case(r, R, H, A, member, n=16):
    c = _random_round_case(r, R, 3, A, n=n)
    c["H"] = H
    c["replica"] = int(r.integers(0, H))
    c["hsdp_scale"] = 1.0 / H
    c["member"] = member
    c["replica_wires"] = [None if k == c["replica"] else random_bf16(r, n, std=10.0 ** r.uniform(-4, -1))
                          for a in range(A) for k in range(H)]
    c["bcast"] = (c["p0"] + r.standard_normal(n) * 1e-3).astype(np.float32)
    return c


def check_hsdp_against_brute_force(orc, hp, c):
    n = c["p0"].size
    master, m, v = c["p0"].copy(), c["m0"].copy(), c["v0"].copy()
    work = torch_bf16_bits(master)
    ss = orc.round_hsdp(c["seg_off"], c["seg_decay"], c["R"], c["H"], c["replica"], c["hsdp_scale"],
                        c["member"], c["G"], c["A"], c["self_group"], c["grad_scale"], hp, c["step0"],
                        c["weights"], c["grads"], c["replica_wires"], c["replicas"], c["bcast"],
                        master, m, v, work, want_sumsq=True)
    tag = "HSDP R=%d H=%d A=%d member=%d" % (c["R"], c["H"], c["A"], c["member"])
    # tier 1 and 2 per step, float64 with bounds; the own wire shard is the
    # oracle's where its bf16 rounding is ambiguous within the bound
    gsteps = []
    for a in range(c["A"]):
        ga = c["grads"][a * c["R"]:(a + 1) * c["R"]]
        g1, e1 = _bf_reduce(ga, c["grad_scale"])
        if c["H"] == 1:
            gsteps.append((g1, e1))
            continue
        own, _ = _resolve_bf16(g1, e1 + TINY, orc.shard_reduce_wire(ga, c["grad_scale"]))
        wires = [own if k == c["replica"] else c["replica_wires"][a * c["H"] + k]
                 for k in range(c["H"])]
        gsteps.append(_bf_reduce(wires, c["hsdp_scale"]))
    (p, ep), (mm, em), (vv, ev) = _bf_steps(hp, c["seg_off"], c["seg_decay"], c["step0"], gsteps,
                                            c["p0"], c["m0"], c["v0"])
    _check_close("hsdp m " + tag, m, mm, em)
    _check_close("hsdp v " + tag, v, vv, ev)
    if c["member"]:
        mw, mmm, mv = c["p0"].copy(), c["m0"].copy(), c["v0"].copy()
        ww = torch_bf16_bits(mw)
        # the oracle's own working copy after the steps, for ambiguous roundings
        for a in range(c["A"]):
            g = orc.shard_reduce(c["grads"][a * c["R"]:(a + 1) * c["R"]], c["grad_scale"]) if c["H"] == 1 else \
                orc.shard_reduce([orc.shard_reduce_wire(c["grads"][a * c["R"]:(a + 1) * c["R"]], c["grad_scale"])
                                  if k == c["replica"] else c["replica_wires"][a * c["H"] + k]
                                  for k in range(c["H"])], c["hsdp_scale"])
            orc.adamw_step(c["seg_off"], c["seg_decay"], hp, c["step0"] + a, g, mw, mmm, mv, ww)
        own, _ = _resolve_bf16(p, ep, ww)
        reps = [own if k == c["self_group"] else c["replicas"][k] for k in range(c["G"])]
        xbar, ex = _bf_fedavg(c["weights"], reps)
        _check_close("hsdp master " + tag, master, xbar, ex)
    else:
        assert np.array_equal(master.view(np.uint32), c["bcast"].view(np.uint32)), "bcast master " + tag
    assert np.array_equal(work, torch_bf16_bits(master)), "hsdp working " + tag
    off = c["seg_off"]
    for a, (g, eg) in enumerate(gsteps):
        for s_ in range(off.size - 1):
            sl = slice(off[s_], off[s_ + 1])
            want = np.sum(g[sl] ** 2)
            bound = np.sum(2 * np.abs(g[sl]) * eg[sl] + eg[sl] ** 2) * 2 + 1e-12 * want + TINY
            assert abs(ss[a, s_] - want) <= bound, "hsdp seg_sumsq " + tag


def pin_hsdp_round_brute_force_16(orc):
    """Two-tier rounds for R in {1..3}, H in {1..4}, A in {1, 2}, as a
    FedAvg member and as a broadcast receiver."""
    r = rng(17)
    for hp in (STD_HP, BIG_HP):
        for R in (1, 2, 3):
            for H in (1, 2, 3, 4):
                for A in (1, 2):
                    for member in (1, 0):
                        check_hsdp_against_brute_force(orc, hp, _random_hsdp_case(r, R, H, A, member))


def pin_hsdp_one_replica_is_fsdp(orc):
    """Section 4.2: FL+HSDP with one replica per group is FL+FSDP."""
    r = rng(18)
    c = _random_round_case(r, 4, 3, 3, n=5000)
    outs = []
    for hsdp in (False, True):
        master, m, v = c["p0"].copy(), c["m0"].copy(), c["v0"].copy()
        work = torch_bf16_bits(master)
        if hsdp:
            orc.round_hsdp(c["seg_off"], c["seg_decay"], 4, 1, 0, 1.0, 1, 3, 3, c["self_group"],
                           c["grad_scale"], STD_HP, c["step0"], c["weights"], c["grads"], [None] * 3,
                           c["replicas"], None, master, m, v, work)
        else:
            orc.round(c["seg_off"], c["seg_decay"], 4, 3, 3, c["self_group"], c["grad_scale"],
                      STD_HP, c["step0"], c["weights"], c["grads"], c["replicas"], master, m, v, work)
        outs.append((master, m, v, work))
    for x, y in zip(*outs):
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), "H = 1 differs from FSDP"


# ---- outer optimiser (FedOpt / FedMom with Nesterov momentum) --------------

OUTER_HP = [dict(lr=0.7, momentum=0.9, nesterov=True), dict(lr=1.3, momentum=0.5, nesterov=False),
            dict(lr=0.7, momentum=0.0, nesterov=True)]


def _bf_outer(oh, prev, eprev, buf, ebuf, xbar, ex):
    """float64 outer step with propagated bounds on the binary32 evaluation."""
    eta, mu = float(np.float32(oh["lr"])), float(np.float32(oh["momentum"]))
    delta = prev - xbar
    ed = eprev + ex + U * (np.abs(delta) + eprev + ex)
    b = mu * buf + delta
    eb = mu * ebuf + ed + U * mu * (np.abs(buf) + ebuf) + U * (np.abs(b) + mu * ebuf + ed)
    if oh.get("nesterov", True):
        d = delta + mu * b
        e_d = ed + mu * eb + U * mu * (np.abs(b) + eb) + U * (np.abs(d) + ed + mu * eb)
    else:
        d, e_d = b, eb
    p = prev - eta * d
    ep = eprev + eta * e_d + U * eta * (np.abs(d) + e_d) + U * (np.abs(p) + eprev + eta * e_d)
    return p, 2 * ep + TINY, b, 2 * eb + TINY


def pin_outer_vs_torch_sgd(orc):
    """Four outer steps against torch.optim.SGD (momentum, dampening 0,
    Nesterov or not) run in float64 on the outer gradient prev - average."""
    r = rng(19)
    for oh in OUTER_HP:
        n, G = 3000, 4
        prev = (r.standard_normal(n) * 0.02).astype(np.float32)
        buf = np.zeros(n, np.float32)
        theta = torch.tensor(prev.astype(np.float64), requires_grad=True)
        opt = torch.optim.SGD([theta], lr=float(np.float32(oh["lr"])),
                              momentum=float(np.float32(oh["momentum"])), dampening=0.0,
                              nesterov=bool(oh["nesterov"] and oh["momentum"] > 0),
                              weight_decay=0.0)
        p64, ep = prev.astype(np.float64), np.zeros(n)
        b64, eb = np.zeros(n), np.zeros(n)
        for rnd in range(4):
            reps = [torch_bf16_bits((prev + r.standard_normal(n) * 1e-3).astype(np.float32))
                    for _ in range(G)]
            w = r.uniform(0.5, 3.0, G).astype(np.float32)
            master, work = orc.fedopt(reps, w, oh, prev, buf)
            xbar, ex = _bf_fedavg(w, reps)
            theta.grad = torch.tensor(theta.detach().numpy() - xbar)
            opt.step()
            p64, ep, b64, eb = _bf_outer(oh, p64, ep, b64, eb, xbar, ex)
            tag = "outer %s round %d" % (oh, rnd)
            _check_close(tag + " torch param", prev, theta.detach().numpy(), ep)
            if oh["momentum"] > 0:
                tb = opt.state[theta]["momentum_buffer"].numpy()
                _check_close(tag + " torch buffer", buf, tb, eb)
            assert np.array_equal(master.view(np.uint32), prev.view(np.uint32)), tag + " master"
            assert np.array_equal(work, torch_bf16_bits(master)), tag + " working"


def pin_outer_unit_lr_no_momentum_is_fedavg(orc):
    """eta = 1, mu = 0: p = prev - (prev - xbar); where prev and xbar are
    within a factor of 2 both subtractions are exact (Sterbenz), so master is
    FedAvg's bitwise; elsewhere within the two roundings' bound."""
    r = rng(20)
    n, G = 5000, 3
    prev = (r.standard_normal(n) * 0.02).astype(np.float32)
    reps = [torch_bf16_bits((prev + r.standard_normal(n) * 1e-4).astype(np.float32))
            for _ in range(G)]
    w = np.array([1.0, 2.0, 3.0], np.float32)
    fa, _ = orc.fedavg(reps, w)
    p, b = prev.copy(), np.zeros(n, np.float32)
    master, _ = orc.fedopt(reps, w, dict(lr=1.0, momentum=0.0, nesterov=True), p, b)
    exact = (np.sign(prev) == np.sign(fa)) & (np.abs(fa) <= 2 * np.abs(prev)) & \
        (np.abs(prev) <= 2 * np.abs(fa))
    assert exact.mean() > 0.9
    assert np.array_equal(master[exact].view(np.uint32), fa[exact].view(np.uint32)), "not FedAvg"
    d64 = prev.astype(np.float64) - fa.astype(np.float64)
    bound = 2 * U * (np.abs(d64) + np.abs(fa.astype(np.float64))) + TINY
    _check_close("eta1 mu0", master[~exact], fa[~exact].astype(np.float64), bound[~exact])


def pin_outer_fixed_point(orc):
    """Replicas equal to the global model and no momentum: nothing moves."""
    r = rng(21)
    x = random_bf16(r, 4000, std=0.02)
    prev = bf16_decode(x).astype(np.float32)
    buf = np.zeros(4000, np.float32)
    master, work = orc.fedopt([x, x, x], np.array([1, 1, 2], np.float32),
                              dict(lr=0.7, momentum=0.9, nesterov=True), prev, buf)
    assert np.array_equal(master, bf16_decode(x).astype(np.float32)), "fixed point moved"
    assert not buf.any() and np.array_equal(work, x)


def pin_round_outer_brute_force_16(orc):
    """A local steps then the outer step, every (R, G, A) in {1..3}^3, two
    outer settings, two rounds in a row (prev and buf carried over)."""
    r = rng(22)
    for oh in OUTER_HP[:2]:
        for R in (1, 2, 3):
            for G in (1, 2, 3):
                for A in (1, 2, 3):
                    c = _random_round_case(r, R, G, A)
                    n = c["p0"].size
                    prev = (c["p0"] + r.standard_normal(n) * 1e-3).astype(np.float32)
                    buf = (r.standard_normal(n) * 1e-4).astype(np.float32)
                    p64, ep = prev.astype(np.float64), np.zeros(n)
                    b64, eb = buf.astype(np.float64), np.zeros(n)
                    master, m, v = c["p0"].copy(), c["m0"].copy(), c["v0"].copy()
                    work = torch_bf16_bits(master)
                    orc.round_outer(c["seg_off"], c["seg_decay"], R, G, A, c["self_group"],
                                    c["grad_scale"], STD_HP, c["step0"], c["weights"], oh,
                                    c["grads"], c["replicas"], prev, buf, master, m, v, work)
                    # float64 local steps; own bf16 copy from the oracle where ambiguous
                    mw, mm, mv = c["p0"].copy(), c["m0"].copy(), c["v0"].copy()
                    ww = torch_bf16_bits(mw)
                    for a in range(A):
                        g = orc.shard_reduce(c["grads"][a * R:(a + 1) * R], c["grad_scale"])
                        orc.adamw_step(c["seg_off"], c["seg_decay"], STD_HP, c["step0"] + a, g,
                                       mw, mm, mv, ww)
                    gsteps = [_bf_reduce(c["grads"][a * R:(a + 1) * R], c["grad_scale"])
                              for a in range(A)]
                    (p, e_p), (mm64, em), (vv64, ev) = _bf_steps(
                        STD_HP, c["seg_off"], c["seg_decay"], c["step0"], gsteps, c["p0"],
                        c["m0"], c["v0"])
                    own, _ = _resolve_bf16(p, e_p, ww)
                    reps = [own if k == c["self_group"] else c["replicas"][k] for k in range(G)]
                    xbar, ex = _bf_fedavg(c["weights"], reps)
                    p64, ep, b64, eb = _bf_outer(oh, p64, ep, b64, eb, xbar, ex)
                    tag = "round_outer %s R=%d G=%d A=%d" % (oh, R, G, A)
                    _check_close(tag + " master", master, p64, ep)
                    _check_close(tag + " prev", prev, p64, ep)
                    _check_close(tag + " buf", buf, b64, eb)
                    _check_close(tag + " m", m, mm64, em)
                    assert np.array_equal(work, torch_bf16_bits(master)), tag


# ---- learning-rate schedule (cosine decay with warm-up) ----------------------

def pin_lr_cosine_vs_transformers(orc):
    """Every step of transformers' cosine-with-warm-up schedules (the lr that
    optimiser step t uses is the scheduler's value after t - 1 steps)."""
    import transformers

    for T, W, lr_max, lr_min in ((64, 7, 3e-4, 0.0), (1000, 100, 1e-3, 1e-5), (10, 0, 0.5, 0.0),
                                 (5, 5, 2e-4, 0.0)):
        base = float(np.float32(lr_max))
        p = torch.nn.Parameter(torch.zeros(1))
        opt = torch.optim.SGD([p], lr=base)
        if lr_min:
            sch = transformers.get_cosine_with_min_lr_schedule_with_warmup(
                opt, W, T, min_lr_rate=float(np.float32(lr_min)) / base)
        else:
            sch = transformers.get_cosine_schedule_with_warmup(opt, W, T)
        for t in range(1, T + 3):
            want = np.float32(opt.param_groups[0]["lr"])
            got = np.float32(orc.lr_cosine(t, T, W, lr_max, lr_min))
            assert got == want, "lr at step %d of (T=%d, W=%d): %r vs %r" % (t, T, W, got, want)
            opt.step()
            sch.step()


def pin_lr_cosine_closed_forms(orc):
    T, W, lr = 100, 10, np.float32(3e-4)
    assert orc.lr_cosine(1, T, W, lr) == 0.0, "warm-up starts at 0"
    assert np.float32(orc.lr_cosine(W + 1, T, W, lr)) == lr, "peak after warm-up"
    mid = W + 1 + (T - W) // 2
    assert abs(orc.lr_cosine(mid, T, W, lr) - lr / 2) <= 1e-3 * lr, "half way down"
    vals = [orc.lr_cosine(t, T, W, lr) for t in range(W + 1, T + 1)]
    assert all(a >= b for a, b in zip(vals, vals[1:])), "cosine part not decreasing"
    ramp = [orc.lr_cosine(t, T, W, lr) for t in range(1, W + 2)]
    assert all(b > a for a, b in zip(ramp, ramp[1:])), "warm-up not increasing"


def pin_round_step_lr_brute_force(orc):
    """A round whose local steps use different learning rates (a schedule)."""
    r = rng(23)
    for A in (2, 3):
        c = _random_round_case(r, 2, 2, A, n=64)
        lrs = [float(np.float32(x)) for x in r.uniform(1e-4, 5e-2, A)]
        master, m, v = c["p0"].copy(), c["m0"].copy(), c["v0"].copy()
        work = torch_bf16_bits(master)
        orc.round(c["seg_off"], c["seg_decay"], 2, 2, A, c["self_group"], c["grad_scale"], BIG_HP,
                  c["step0"], c["weights"], c["grads"], c["replicas"], master, m, v, work,
                  step_lr=lrs)
        gsteps = [_bf_reduce(c["grads"][a * 2:(a + 1) * 2], c["grad_scale"]) for a in range(A)]
        (p, ep), (mm, em), (vv, ev) = _bf_steps(BIG_HP, c["seg_off"], c["seg_decay"], c["step0"],
                                                gsteps, c["p0"], c["m0"], c["v0"], lrs=lrs)
        _check_close("step_lr m", m, mm, em)
        _check_close("step_lr v", v, vv, ev)
        mw, mmm, mv = c["p0"].copy(), c["m0"].copy(), c["v0"].copy()
        ww = torch_bf16_bits(mw)
        for a in range(A):
            g = orc.shard_reduce(c["grads"][a * 2:(a + 1) * 2], c["grad_scale"])
            orc.adamw_step(c["seg_off"], c["seg_decay"], dict(BIG_HP, lr=lrs[a]), c["step0"] + a,
                           g, mw, mmm, mv, ww)
        own, _ = _resolve_bf16(p, ep, ww)
        reps = [own if k == c["self_group"] else c["replicas"][k] for k in range(2)]
        xbar, ex = _bf_fedavg(c["weights"], reps)
        _check_close("step_lr master", master, xbar, ex)


# ---- global-norm gradient clipping -------------------------------------------

def pin_clip_vs_torch(orc):
    """Coefficient and clipped gradient against torch.nn.utils.clip_grad_norm_
    in float64, including a norm small enough that its 1e-6 guard matters."""
    r = rng(24)
    for scale, max_norm in ((1e-3, 0.05), (1e-3, 100.0), (1e-9, 1e-10), (0.3, 1.0)):
        g = (r.standard_normal(20000) * scale).astype(np.float32)
        t = torch.nn.Parameter(torch.zeros(g.size, dtype=torch.float64))
        t.grad = torch.tensor(g.astype(np.float64))
        total_norm = float(torch.nn.utils.clip_grad_norm_([t], max_norm))
        total = orc.total_sumsq(g)
        assert abs(total - total_norm ** 2) <= 1e-12 * total_norm ** 2 + 1e-300, "sum of squares"
        coef = orc.clip_coef(total, max_norm)
        want = min(1.0, float(np.float32(max_norm)) / (total_norm + 1e-6))
        assert abs(coef - want) <= 2 * U * want, "clip coefficient %r vs %r" % (coef, want)
        clipped = g * np.float32(coef)
        _check_close("clipped g", clipped, t.grad.numpy(), 4 * U * np.abs(t.grad.numpy()) + TINY)


def pin_clip_nonfinite_norm_vs_torch(orc):
    """A NaN or infinite gradient norm: the coefficient and the clipped
    gradient are torch.nn.utils.clip_grad_norm_'s (NaN everywhere for a NaN
    norm; zero, and NaN at an infinite entry, for an infinite norm)."""
    for bad in (np.nan, np.inf):
        g = np.array([1e-3, -2e-3, bad, 4e-3], np.float32)
        t = torch.nn.Parameter(torch.zeros(g.size, dtype=torch.float64))
        t.grad = torch.tensor(g.astype(np.float64))
        torch.nn.utils.clip_grad_norm_([t], 1.0)
        coef = orc.clip_coef(orc.total_sumsq(g), 1.0)
        clipped = (g * np.float32(coef)).astype(np.float64)
        want = t.grad.numpy()
        assert np.array_equal(np.isnan(clipped), np.isnan(want)), (bad, clipped, want)
        fin = ~np.isnan(want)
        assert np.array_equal(clipped[fin], want[fin]), (bad, clipped, want)


def _bf_clip(gsteps, max_norm):
    """Clipped per-step (g, bound) in float64 from unclipped ones."""
    out = []
    M = float(np.float32(max_norm))
    for g, eg in gsteps:
        T = np.sum(g * g)
        dT = np.sum(2 * np.abs(g) * eg + eg * eg) + 1e-15 * T
        c = min(1.0, M / (np.sqrt(T) + 1e-6))
        ec = c * (dT / max(T, 1e-300) / 2 + 2 * U) + 1e-300
        gc = g * c
        out.append((gc, eg * c + np.abs(g) * ec + U * np.abs(gc)))
    return out


def pin_round_clipped_brute_force(orc):
    """Rounds with clipping active (norm above max) and inactive."""
    r = rng(25)
    for R, A, max_norm in ((2, 2, 1e-3), (3, 3, 5e-4), (2, 2, 1e6)):
        c = _random_round_case(r, R, 2, A, n=48)
        master, m, v = c["p0"].copy(), c["m0"].copy(), c["v0"].copy()
        work = torch_bf16_bits(master)
        ss = orc.round(c["seg_off"], c["seg_decay"], R, 2, A, c["self_group"], c["grad_scale"],
                       BIG_HP, c["step0"], c["weights"], c["grads"], c["replicas"], master, m, v,
                       work, want_sumsq=True, max_grad_norm=max_norm)
        g0 = [_bf_reduce(c["grads"][a * R:(a + 1) * R], c["grad_scale"]) for a in range(A)]
        gsteps = _bf_clip(g0, max_norm)
        (p, ep), (mm, em), (vv, ev) = _bf_steps(BIG_HP, c["seg_off"], c["seg_decay"], c["step0"],
                                                gsteps, c["p0"], c["m0"], c["v0"])
        tag = "clip R=%d A=%d max=%g" % (R, A, max_norm)
        _check_close(tag + " m", m, mm, em)
        _check_close(tag + " v", v, vv, ev)
        off = c["seg_off"]
        for a, (g, eg) in enumerate(g0):   # per-segment sums are of the unclipped g
            for s_ in range(off.size - 1):
                sl = slice(off[s_], off[s_ + 1])
                want = np.sum(g[sl] ** 2)
                bound = np.sum(2 * np.abs(g[sl]) * eg[sl] + eg[sl] ** 2) * 2 + 1e-12 * want + TINY
                assert abs(ss[a, s_] - want) <= bound, tag + " seg_sumsq"


def pin_grad_total_streams(orc):
    """The streamed whole-shard total equals a float64 sum of the squares of
    the reduced gradient, and chunking it changes nothing."""
    r = rng(27)
    grads = [random_bf16(r, 10000, 1e-3) for _ in range(3)]
    whole = orc.grad_total(grads, 1.0 / 3)
    g = orc.shard_reduce(grads, 1.0 / 3).astype(np.float64)
    assert abs(whole - np.sum(g * g)) <= 1e-12 * whole
    acc = 0.0
    for lo in range(0, 10000, 3333):
        acc = orc.grad_total([x[lo:lo + 3333] for x in grads], 1.0 / 3, acc)
    assert acc == whole, "chunked total differs"


def pin_clip_inactive_is_bitwise_unclipped(orc):
    r = rng(26)
    c = _random_round_case(r, 3, 2, 3, n=4000)
    outs = []
    for mx in (0.0, 1e9):
        master, m, v = c["p0"].copy(), c["m0"].copy(), c["v0"].copy()
        work = torch_bf16_bits(master)
        orc.round(c["seg_off"], c["seg_decay"], 3, 2, 3, c["self_group"], c["grad_scale"], STD_HP,
                  c["step0"], c["weights"], c["grads"], c["replicas"], master, m, v, work,
                  max_grad_norm=mx)
        outs.append((master, m, v, work))
    for x, y in zip(*outs):
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), "coef 1 changed the round"


ALL_PINS = [
    pin_bf16_decode_all_patterns,
    pin_bf16_encode_matches_torch,
    pin_bf16_encode_nan,
    pin_reduce_vs_float64_sum,
    pin_reduce_identical_peers_exact,
    pin_seg_sumsq_vs_numpy,
    pin_adamw_vs_torch_float64,
    pin_adamw_first_step_closed_form,
    pin_adamw_zero_grad,
    pin_adamw_lr_zero,
    pin_fedavg_identical_replicas,
    pin_fedavg_two_group_mean,
    pin_fedavg_vs_float64_average,
    pin_fedavg_weight_scale_invariance,
    pin_golden_hand_cases,
    pin_round_brute_force_16,
    pin_round_single_step_single_group,
    pin_round_uses_own_working_copy,
    pin_reduce_wire_vs_float64,
    pin_broadcast_recv,
    pin_hsdp_round_brute_force_16,
    pin_hsdp_one_replica_is_fsdp,
    pin_outer_vs_torch_sgd,
    pin_outer_unit_lr_no_momentum_is_fedavg,
    pin_outer_fixed_point,
    pin_round_outer_brute_force_16,
    pin_lr_cosine_vs_transformers,
    pin_lr_cosine_closed_forms,
    pin_round_step_lr_brute_force,
    pin_clip_vs_torch,
    pin_round_clipped_brute_force,
    pin_clip_inactive_is_bitwise_unclipped,
    pin_grad_total_streams,
    pin_clip_nonfinite_norm_vs_torch,
]
