"""Python face of the CPU oracle (liboracle.so).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the CPU-baseline
leg of the benchmark use this; the product path never does.  The oracle's
arithmetic lives in oracle.c; this module only marshals numpy arrays.
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# ORACLE_LIB names another build of oracle.c to load (the sanitizer test's)
_LIB_PATH = os.environ.get("ORACLE_LIB") or os.path.join(HERE, "liboracle.so")

_P = ctypes.c_void_p


class Outer(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("momentum", ctypes.c_float), ("nesterov", ctypes.c_int)]


def outer(oh):
    return Outer(oh["lr"], oh["momentum"], 1 if oh.get("nesterov", True) else 0)


class Hparams(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float)]


def _declare(lib):
    lib.orc_bf16_to_f32.argtypes = [ctypes.c_uint16]
    lib.orc_bf16_to_f32.restype = ctypes.c_float
    lib.orc_f32_to_bf16.argtypes = [ctypes.c_float]
    lib.orc_f32_to_bf16.restype = ctypes.c_uint16
    lib.orc_f32_to_bf16_array.argtypes = [ctypes.c_int64, _P, _P]
    lib.orc_bf16_to_f32_array.argtypes = [ctypes.c_int64, _P, _P]
    lib.orc_shard_reduce.argtypes = [ctypes.c_int64, ctypes.c_int, _P, ctypes.c_float, _P]
    lib.orc_seg_sumsq.argtypes = [ctypes.c_int64, _P, _P, _P]
    lib.orc_adamw_step.argtypes = [ctypes.c_int64, _P, _P, ctypes.POINTER(Hparams),
                                   ctypes.c_int64, _P, _P, _P, _P, _P]
    lib.orc_fedavg.argtypes = [ctypes.c_int64, ctypes.c_int, _P, _P, _P, _P]
    lib.orc_round.argtypes = [ctypes.c_int64, _P, _P, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                              ctypes.c_int, ctypes.c_float, ctypes.POINTER(Hparams),
                              ctypes.c_int64, _P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_float,
                              _P]
    lib.orc_lr_cosine.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_float,
                                  ctypes.c_float]
    lib.orc_lr_cosine.restype = ctypes.c_float
    lib.orc_total_sumsq.argtypes = [ctypes.c_int64, _P]
    lib.orc_total_sumsq.restype = ctypes.c_double
    lib.orc_clip_coef.argtypes = [ctypes.c_double, ctypes.c_float]
    lib.orc_clip_coef.restype = ctypes.c_float
    lib.orc_grad_total.argtypes = [ctypes.c_int64, ctypes.c_int, _P, ctypes.c_float,
                                   ctypes.c_double]
    lib.orc_grad_total.restype = ctypes.c_double
    lib.orc_shard_reduce_wire.argtypes = [ctypes.c_int64, ctypes.c_int, _P, ctypes.c_float, _P]
    lib.orc_broadcast_recv.argtypes = [ctypes.c_int64, _P, _P, _P]
    lib.orc_round_hsdp.argtypes = [ctypes.c_int64, _P, _P, ctypes.c_int, ctypes.c_int,
                                   ctypes.c_int, ctypes.c_float, ctypes.c_int, ctypes.c_int,
                                   ctypes.c_int, ctypes.c_int, ctypes.c_float,
                                   ctypes.POINTER(Hparams), ctypes.c_int64, _P, _P, _P, _P, _P,
                                   _P, _P, _P, _P, _P, _P, ctypes.c_float, _P]
    lib.orc_fedopt.argtypes = [ctypes.c_int64, ctypes.c_int, _P, _P, ctypes.POINTER(Outer), _P,
                               _P, _P, _P]
    lib.orc_round_outer.argtypes = [ctypes.c_int64, _P, _P, ctypes.c_int, ctypes.c_int,
                                    ctypes.c_int, ctypes.c_int, ctypes.c_float,
                                    ctypes.POINTER(Hparams), ctypes.c_int64, _P,
                                    ctypes.POINTER(Outer), _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                    _P, ctypes.c_float, _P]
    return lib


_lib = None


def lib(path=None):
    """The oracle library; `path` loads another build (a test's mutant)."""
    global _lib
    if path is not None:
        return _declare(ctypes.CDLL(path))
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError("oracle not built: %s missing (run oracle/build.py)" % _LIB_PATH)
        _lib = _declare(ctypes.CDLL(_LIB_PATH))
    return _lib


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


def _ptr_array(arrays):
    return (ctypes.c_void_p * len(arrays))(*[a.ctypes.data for a in arrays])


def _lr_arr(step_lr, A):
    """The per-step learning rates as a float32 array (or None); the caller
    holds it for the duration of the oracle call."""
    if step_lr is None:
        return None
    a = np.ascontiguousarray(step_lr, dtype=np.float32)
    assert a.size == A, "step_lr needs one value per local step"
    return a


def _tot_arr(totals, A):
    """The per-step whole-shard sums of squares as a float64 array (or
    None); the caller holds it for the duration of the oracle call."""
    if totals is None:
        return None
    a = np.ascontiguousarray(totals, dtype=np.float64)
    assert a.size == A, "clip_totals needs one value per local step"
    return a


def _ptr(a):
    return None if a is None else a.ctypes.data


def hparams(hp):
    return Hparams(hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["weight_decay"])


class Oracle:
    """Numpy wrappers over one oracle build."""

    def __init__(self, path=None):
        self.L = lib(path)

    def f32_to_bf16(self, x):
        x = _c(x, np.float32)
        out = np.empty(x.shape, np.uint16)
        self.L.orc_f32_to_bf16_array(x.size, x.ctypes.data, out.ctypes.data)
        return out

    def bf16_to_f32(self, x):
        x = _c(x, np.uint16)
        out = np.empty(x.shape, np.float32)
        self.L.orc_bf16_to_f32_array(x.size, x.ctypes.data, out.ctypes.data)
        return out

    def shard_reduce(self, grads, grad_scale):
        grads = [_c(g, np.uint16) for g in grads]
        n = grads[0].size
        out = np.empty(n, np.float32)
        rc = self.L.orc_shard_reduce(n, len(grads), _ptr_array(grads), grad_scale,
                                     out.ctypes.data)
        if rc:
            raise ValueError("orc_shard_reduce: %d" % rc)
        return out

    def seg_sumsq(self, seg_off, g):
        seg_off = _c(seg_off, np.int64)
        g = _c(g, np.float32)
        out = np.empty(seg_off.size - 1, np.float64)
        rc = self.L.orc_seg_sumsq(seg_off.size - 1, seg_off.ctypes.data, g.ctypes.data,
                                  out.ctypes.data)
        if rc:
            raise ValueError("orc_seg_sumsq: %d" % rc)
        return out

    def adamw_step(self, seg_off, seg_decay, hp, t, g, master, m, v, working=None):
        """In place on master, m, v (float32) and working (uint16, optional)."""
        seg_off = _c(seg_off, np.int64)
        seg_decay = _c(seg_decay, np.uint8)
        g = _c(g, np.float32)
        for a in (master, m, v):
            assert a.dtype == np.float32 and a.flags.c_contiguous
        h = hparams(hp)
        wp = None if working is None else working.ctypes.data
        rc = self.L.orc_adamw_step(seg_off.size - 1, seg_off.ctypes.data, seg_decay.ctypes.data,
                                   ctypes.byref(h), t, g.ctypes.data, master.ctypes.data,
                                   m.ctypes.data, v.ctypes.data, wp)
        if rc:
            raise ValueError("orc_adamw_step: %d" % rc)

    def fedavg(self, replicas, weights, master_out=None, working_out=None):
        replicas = [_c(r, np.uint16) for r in replicas]
        n = replicas[0].size
        w = _c(weights, np.float32)
        master_out = np.empty(n, np.float32) if master_out is None else master_out
        working_out = np.empty(n, np.uint16) if working_out is None else working_out
        rc = self.L.orc_fedavg(n, len(replicas), _ptr_array(replicas), w.ctypes.data,
                               master_out.ctypes.data, working_out.ctypes.data)
        if rc:
            raise ValueError("orc_fedavg: %d" % rc)
        return master_out, working_out

    def shard_reduce_wire(self, grads, grad_scale):
        grads = [_c(g, np.uint16) for g in grads]
        n = grads[0].size
        out = np.empty(n, np.uint16)
        rc = self.L.orc_shard_reduce_wire(n, len(grads), _ptr_array(grads), grad_scale,
                                          out.ctypes.data)
        if rc:
            raise ValueError("orc_shard_reduce_wire: %d" % rc)
        return out

    def broadcast_recv(self, recv, master, working):
        recv = _c(recv, np.float32)
        rc = self.L.orc_broadcast_recv(recv.size, recv.ctypes.data, master.ctypes.data,
                                       working.ctypes.data)
        if rc:
            raise ValueError("orc_broadcast_recv: %d" % rc)

    def round_hsdp(self, seg_off, seg_decay, R, H, replica, hsdp_scale, member, G, A,
                   self_group, grad_scale, hp, step0, weights, grads, replica_wires, replicas,
                   bcast, master, m, v, working, want_sumsq=False, step_lr=None,
                   max_grad_norm=0.0, clip_totals=None):
        """One FL+HSDP round in place.  replica_wires: A*H arrays (entry
        a*H + replica ignored, may be None); replicas: G arrays or None
        (member only); bcast: fp32 array (non-member only)."""
        seg_off = _c(seg_off, np.int64)
        seg_decay = _c(seg_decay, np.uint8)
        n_seg = seg_off.size - 1
        n = int(seg_off[-1])
        dummy = np.zeros(max(n, 1), np.uint16)
        grads = [_c(g, np.uint16) for g in grads]
        wires = [dummy if x is None else _c(x, np.uint16) for x in (replica_wires or [])]
        reps = [working if x is None else _c(x, np.uint16) for x in (replicas or [])]
        w = _c(weights if weights is not None else [1.0], np.float32)
        bc = None if bcast is None else _c(bcast, np.float32)
        h = hparams(hp)
        lr_a, tot_a = _lr_arr(step_lr, A), _tot_arr(clip_totals, A)
        ss = np.empty(A * n_seg, np.float64) if want_sumsq else None
        rc = self.L.orc_round_hsdp(n_seg, seg_off.ctypes.data, seg_decay.ctypes.data, R, H, replica,
                                   hsdp_scale, 1 if member else 0, G, A, self_group, grad_scale,
                                   ctypes.byref(h), step0, w.ctypes.data, _ptr_array(grads),
                                   _ptr_array(wires) if wires else None,
                                   _ptr_array(reps) if reps else None,
                                   None if bc is None else bc.ctypes.data, master.ctypes.data,
                                   m.ctypes.data, v.ctypes.data, working.ctypes.data,
                                   None if ss is None else ss.ctypes.data, _ptr(lr_a),
                                   max_grad_norm, _ptr(tot_a))
        if rc:
            raise ValueError("orc_round_hsdp: %d" % rc)
        return None if ss is None else ss.reshape(A, n_seg)

    def fedopt(self, replicas, weights, oh, prev, buf, master_out=None, working_out=None):
        """Outer step in place on prev and buf; returns (master, working)."""
        replicas = [_c(r, np.uint16) for r in replicas]
        n = replicas[0].size
        w = _c(weights, np.float32)
        o = outer(oh)
        master_out = np.empty(n, np.float32) if master_out is None else master_out
        working_out = np.empty(n, np.uint16) if working_out is None else working_out
        rc = self.L.orc_fedopt(n, len(replicas), _ptr_array(replicas), w.ctypes.data,
                               ctypes.byref(o), prev.ctypes.data, buf.ctypes.data,
                               master_out.ctypes.data, working_out.ctypes.data)
        if rc:
            raise ValueError("orc_fedopt: %d" % rc)
        return master_out, working_out

    def round_outer(self, seg_off, seg_decay, R, G, A, self_group, grad_scale, hp, step0,
                    weights, oh, grads, replicas, prev, buf, master, m, v, working,
                    want_sumsq=False, step_lr=None, max_grad_norm=0.0, clip_totals=None):
        seg_off = _c(seg_off, np.int64)
        seg_decay = _c(seg_decay, np.uint8)
        n_seg = seg_off.size - 1
        grads = [_c(g, np.uint16) for g in grads]
        reps = [working if r is None else _c(r, np.uint16) for r in replicas]
        w = _c(weights, np.float32)
        h = hparams(hp)
        o = outer(oh)
        lr_a, tot_a = _lr_arr(step_lr, A), _tot_arr(clip_totals, A)
        ss = np.empty(A * n_seg, np.float64) if want_sumsq else None
        rc = self.L.orc_round_outer(n_seg, seg_off.ctypes.data, seg_decay.ctypes.data, R, G, A,
                                    self_group, grad_scale, ctypes.byref(h), step0, w.ctypes.data,
                                    ctypes.byref(o), _ptr_array(grads), _ptr_array(reps),
                                    prev.ctypes.data, buf.ctypes.data, master.ctypes.data,
                                    m.ctypes.data, v.ctypes.data, working.ctypes.data,
                                    None if ss is None else ss.ctypes.data, _ptr(lr_a),
                                    max_grad_norm, _ptr(tot_a))
        if rc:
            raise ValueError("orc_round_outer: %d" % rc)
        return None if ss is None else ss.reshape(A, n_seg)

    def total_sumsq(self, g):
        g = _c(g, np.float32)
        return self.L.orc_total_sumsq(g.size, g.ctypes.data)

    def grad_total(self, grads, grad_scale, acc0=0.0):
        grads = [_c(g, np.uint16) for g in grads]
        return self.L.orc_grad_total(grads[0].size, len(grads), _ptr_array(grads), grad_scale,
                                     acc0)

    def clip_coef(self, total_sumsq, max_norm):
        return self.L.orc_clip_coef(total_sumsq, max_norm)

    def lr_cosine(self, t, total_steps, warmup_steps, lr_max, lr_min=0.0):
        return self.L.orc_lr_cosine(t, total_steps, warmup_steps, lr_max, lr_min)

    def round(self, seg_off, seg_decay, R, G, A, self_group, grad_scale, hp, step0, weights,
              grads, replicas, master, m, v, working, want_sumsq=False, step_lr=None,
              max_grad_norm=0.0, clip_totals=None):
        """In place on master, m, v, working.  grads: A*R arrays step-major;
        replicas: G arrays (entry self_group ignored, may be None).
        Returns the A x n_seg per-segment sums of squares, or None."""
        seg_off = _c(seg_off, np.int64)
        seg_decay = _c(seg_decay, np.uint8)
        n_seg = seg_off.size - 1
        grads = [_c(g, np.uint16) for g in grads]
        reps = [working if r is None else _c(r, np.uint16) for r in replicas]
        w = _c(weights, np.float32)
        h = hparams(hp)
        lr_a, tot_a = _lr_arr(step_lr, A), _tot_arr(clip_totals, A)
        ss = np.empty(A * n_seg, np.float64) if want_sumsq else None
        rc = self.L.orc_round(n_seg, seg_off.ctypes.data, seg_decay.ctypes.data, R, G, A,
                              self_group, grad_scale, ctypes.byref(h), step0, w.ctypes.data,
                              _ptr_array(grads), _ptr_array(reps), master.ctypes.data,
                              m.ctypes.data, v.ctypes.data, working.ctypes.data,
                              None if ss is None else ss.ctypes.data, _ptr(lr_a),
                              max_grad_norm, _ptr(tot_a))
        if rc:
            raise ValueError("orc_round: %d" % rc)
        return None if ss is None else ss.reshape(A, n_seg)


def workload_round(orc, w, host, seg_off=None, seg_decay=None, want_sumsq=False,
                   clip_totals=None, step_lr=None):
    """Run the oracle round of workload w (FL+FSDP, FL+HSDP when w.H > 1, or
    the outer step) in place on the host arrays of `host` (a
    synth.buffers.HostInputs or a view of one).  seg_off / seg_decay: the
    layout of the arrays held (default: the workload's whole shard).
    clip_totals: per-step whole-shard sums of squares to clip against when
    the arrays hold only part of the shard.  Returns the per-step
    per-segment sums of squares (A x n_seg, double) or None."""
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
