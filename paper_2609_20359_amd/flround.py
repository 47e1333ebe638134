"""ctypes binding of libflround (include/flround.h).

Argument marshalling only: every step of the path runs in the library's
gfx950 kernels.  Tensors are torch CUDA tensors (bf16 buffers may be
torch.bfloat16 or any 2-byte dtype holding bf16 bits); work is enqueued on
the current torch stream unless `stream` is given.  Every non-OK status
raises FlError.  If the library is missing, importing the symbols raises:
there is no fallback.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# FLROUND_LIB names another build of the library to load (the sanitizer
# test's host-instrumented build)
LIB_PATH = os.environ.get("FLROUND_LIB") or os.path.join(HERE, "libflround.so")

FL_OK = 0
FL_ERR_INVALID = -1
FL_ERR_ALIGN = -2
FL_ERR_LAYOUT = -3
FL_ERR_DEVICE = -4
FL_ERR_HIP = -5
FL_ERR_NOMEM = -6
FL_ERR_SCRATCH = -7
FL_NOALLOC_SCRATCH_BYTES = 32 << 20

FL_MAX_PEERS = 64
FL_MAX_GROUPS = 64

# Every symbol include/flround.h declares.
EXPORTS = ("fl_status_string", "fl_version", "fl_layout_create", "fl_layout_destroy",
           "fl_layout_numel", "fl_layout_num_segments", "fl_fingerprint",
           "fl_layout_fingerprint", "fl_shard_reduce", "fl_adamw_step", "fl_local_step",
           "fl_fedavg", "fl_round", "fl_set_blocks_per_cu", "fl_shard_reduce_wire",
           "fl_broadcast_recv", "fl_round_hsdp", "fl_fedopt", "fl_round_outer",
           "fl_lr_cosine", "fl_grad_sumsq", "fl_local_step_clipped", "fl_round_noalloc",
           "fl_noalloc_workspace_bytes")

_P = ctypes.c_void_p


class FlError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__("%s: %s" % (where, status_string(status)))


class AdamwHparams(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float)]


class RoundCfg(ctypes.Structure):
    _fields_ = [("R", ctypes.c_int), ("G", ctypes.c_int), ("A", ctypes.c_int),
                ("self_group", ctypes.c_int), ("grad_scale", ctypes.c_float),
                ("h", AdamwHparams), ("step0", ctypes.c_int64),
                ("weights", ctypes.POINTER(ctypes.c_float)),
                ("replica_fp", ctypes.POINTER(ctypes.c_uint64)),
                ("phase_events", ctypes.POINTER(ctypes.c_void_p)),
                ("step_lr", ctypes.POINTER(ctypes.c_float)),
                ("max_grad_norm", ctypes.c_float),
                ("grad_scratch", ctypes.c_void_p)]


class OuterHparams(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("momentum", ctypes.c_float), ("nesterov", ctypes.c_int)]


def outer_hparams(oh):
    if isinstance(oh, OuterHparams):
        return oh
    return OuterHparams(oh["lr"], oh["momentum"], 1 if oh.get("nesterov", True) else 0)


class HsdpCfg(ctypes.Structure):
    _fields_ = [("H", ctypes.c_int), ("replica", ctypes.c_int), ("hsdp_scale", ctypes.c_float),
                ("fedavg_member", ctypes.c_int)]


_lib = None


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libflround.so is not built (%s); run "
                               "`python -m paper_2609_20359_amd.build`" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        L.fl_status_string.argtypes = [ctypes.c_int]
        L.fl_status_string.restype = ctypes.c_char_p
        L.fl_version.restype = ctypes.c_int
        L.fl_layout_create.argtypes = [ctypes.c_int64, ctypes.c_int64, _P, _P,
                                       ctypes.POINTER(_P)]
        L.fl_layout_destroy.argtypes = [_P]
        L.fl_layout_numel.argtypes = [_P]
        L.fl_layout_numel.restype = ctypes.c_int64
        L.fl_layout_num_segments.argtypes = [_P]
        L.fl_layout_num_segments.restype = ctypes.c_int64
        L.fl_fingerprint.argtypes = [ctypes.c_int64, ctypes.c_int64, _P, _P]
        L.fl_fingerprint.restype = ctypes.c_uint64
        L.fl_layout_fingerprint.argtypes = [_P]
        L.fl_layout_fingerprint.restype = ctypes.c_uint64
        L.fl_shard_reduce.argtypes = [_P, ctypes.c_int, _P, ctypes.c_float, _P, _P, _P]
        L.fl_adamw_step.argtypes = [_P, ctypes.POINTER(AdamwHparams), ctypes.c_int64, _P, _P,
                                    _P, _P, _P, _P]
        L.fl_local_step.argtypes = [_P, ctypes.POINTER(AdamwHparams), ctypes.c_int64,
                                    ctypes.c_int, _P, ctypes.c_float, _P, _P, _P, _P, _P, _P]
        L.fl_fedavg.argtypes = [_P, ctypes.c_int, _P, _P, _P, _P, _P, _P]
        L.fl_round.argtypes = [_P, ctypes.POINTER(RoundCfg), _P, _P, _P, _P, _P, _P, _P, _P]
        L.fl_round_noalloc.argtypes = [_P, ctypes.POINTER(RoundCfg), _P, _P, _P, _P, _P, _P, _P,
                                       _P]
        L.fl_noalloc_workspace_bytes.argtypes = [_P]
        L.fl_noalloc_workspace_bytes.restype = ctypes.c_size_t
        L.fl_shard_reduce_wire.argtypes = [_P, ctypes.c_int, _P, ctypes.c_float, _P, _P]
        L.fl_broadcast_recv.argtypes = [_P, _P, _P, _P, _P]
        L.fl_round_hsdp.argtypes = [_P, ctypes.POINTER(RoundCfg), ctypes.POINTER(HsdpCfg), _P, _P,
                                    _P, _P, _P, _P, _P, _P, _P, _P, _P]
        L.fl_fedopt.argtypes = [_P, ctypes.c_int, _P, _P, _P, ctypes.POINTER(OuterHparams), _P, _P,
                                _P, _P, _P]
        L.fl_round_outer.argtypes = [_P, ctypes.POINTER(RoundCfg), ctypes.POINTER(OuterHparams),
                                     _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]
        L.fl_grad_sumsq.argtypes = [_P, ctypes.c_int, _P, ctypes.c_float, _P, _P, _P]
        L.fl_local_step_clipped.argtypes = [_P, ctypes.POINTER(AdamwHparams), ctypes.c_int64,
                                            ctypes.c_int, _P, ctypes.c_float, _P, ctypes.c_float,
                                            _P, _P, _P, _P, _P]
        L.fl_lr_cosine.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_float,
                                   ctypes.c_float]
        L.fl_lr_cosine.restype = ctypes.c_float
        L.fl_set_blocks_per_cu.argtypes = [ctypes.c_int]
        L.fl_set_blocks_per_cu.restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(status):
    return lib().fl_status_string(status).decode()


def _check(rc, where):
    if rc != FL_OK:
        raise FlError(rc, where)


_MAX_LIST = 1 << 20


def _buf(t, n, esize, what):
    """Device address of a tensor argument, after checking on the host what
    the kernels assume of it: a contiguous CUDA tensor of exactly n elements
    of esize bytes.  None gives NULL (the library decides whether that is
    allowed); an int is taken as a raw device address."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not getattr(t, "is_cuda", False):
        raise ValueError("%s must be a CUDA tensor" % what)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % what)
    if t.element_size() != esize:
        raise ValueError("%s has %d-byte elements; expected %d" % (what, t.element_size(), esize))
    if t.numel() != n:
        raise ValueError("%s has %d elements; expected %d" % (what, t.numel(), n))
    return t.data_ptr()


def _bufs(ts, count, n, esize, what):
    """Host array of the device addresses of `count` tensors (each checked as
    in _buf).  A shorter list is padded with NULL, which the library rejects
    with FL_ERR_INVALID; a longer one is an error.  When `count` is outside
    what any call accepts, the list is passed as given for the library to
    reject the configuration."""
    ts = list(ts)
    if 1 <= count <= _MAX_LIST:
        if len(ts) > count:
            raise ValueError("%s has %d entries; expected %d" % (what, len(ts), count))
        size = count
    else:
        size = max(len(ts), 1)
    arr = (ctypes.c_void_p * size)()
    for i, t in enumerate(ts):
        arr[i] = _buf(t, n, esize, "%s[%d]" % (what, i))
    return arr


def _host_list(xs, count, ctype, what):
    xs = list(xs)
    if len(xs) != count:
        raise ValueError("%s has %d entries; expected %d" % (what, len(xs), count))
    return (ctype * max(count, 1))(*xs)


def _stream(stream):
    if stream is not None:
        return ctypes.c_void_p(stream if isinstance(stream, int) else stream.cuda_stream)
    import torch

    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def hparams(hp):
    if isinstance(hp, AdamwHparams):
        return hp
    return AdamwHparams(hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["weight_decay"])


def set_blocks_per_cu(n):
    """Cap the streaming kernels' grid at n * CUs (0 = default); returns the
    previous value."""
    return lib().fl_set_blocks_per_cu(int(n))


def fingerprint(seg_offsets, seg_decay=None):
    import numpy as np

    off = np.ascontiguousarray(seg_offsets, dtype=np.int64)
    dec = None if seg_decay is None else np.ascontiguousarray(seg_decay, dtype=np.uint8)
    return lib().fl_fingerprint(int(off[-1]), off.size - 1, off.ctypes.data,
                                None if dec is None else dec.ctypes.data)


class Layout:
    """fl_layout handle: the flat shard's segments and decay flags."""

    def __init__(self, seg_offsets, seg_decay=None):
        import numpy as np

        off = np.ascontiguousarray(seg_offsets, dtype=np.int64)
        dec = None if seg_decay is None else np.ascontiguousarray(seg_decay, dtype=np.uint8)
        h = ctypes.c_void_p()
        rc = lib().fl_layout_create(int(off[-1]), off.size - 1, off.ctypes.data,
                                    None if dec is None else dec.ctypes.data, ctypes.byref(h))
        _check(rc, "fl_layout_create")
        self.handle = h
        self.n = int(off[-1])
        self.n_seg = off.size - 1

    @property
    def fingerprint(self):
        return lib().fl_layout_fingerprint(self.handle)

    def close(self):
        if self.handle:
            lib().fl_layout_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def fl_shard_reduce(layout, peer_grads, grad_scale, grad_out, seg_sumsq=None, stream=None):
    n, R = layout.n, len(peer_grads)
    rc = lib().fl_shard_reduce(layout.handle, R, _bufs(peer_grads, R, n, 2, "peer_grads"),
                               float(grad_scale), _buf(grad_out, n, 4, "grad_out"),
                               _buf(seg_sumsq, layout.n_seg, 4, "seg_sumsq"), _stream(stream))
    _check(rc, "fl_shard_reduce")


def fl_adamw_step(layout, hp, step, grad, master, m, v, working=None, stream=None):
    h = hparams(hp)
    n = layout.n
    rc = lib().fl_adamw_step(layout.handle, ctypes.byref(h), int(step), _buf(grad, n, 4, "grad"),
                             _buf(master, n, 4, "master"), _buf(m, n, 4, "m"),
                             _buf(v, n, 4, "v"), _buf(working, n, 2, "working"), _stream(stream))
    _check(rc, "fl_adamw_step")


def fl_local_step(layout, hp, step, peer_grads, grad_scale, master, m, v, working,
                  seg_sumsq=None, stream=None):
    h = hparams(hp)
    n, R = layout.n, len(peer_grads)
    rc = lib().fl_local_step(layout.handle, ctypes.byref(h), int(step), R,
                             _bufs(peer_grads, R, n, 2, "peer_grads"), float(grad_scale),
                             _buf(master, n, 4, "master"), _buf(m, n, 4, "m"), _buf(v, n, 4, "v"),
                             _buf(working, n, 2, "working"),
                             _buf(seg_sumsq, layout.n_seg, 4, "seg_sumsq"), _stream(stream))
    _check(rc, "fl_local_step")


def fl_fedavg(layout, replicas, weights, master_out, working_out, replica_fp=None, stream=None):
    n, G = layout.n, len(replicas)
    w = _host_list([float(x) for x in weights], G, ctypes.c_float, "weights")
    fp = None if replica_fp is None else _host_list([int(x) for x in replica_fp], G,
                                                    ctypes.c_uint64, "replica_fp")
    rc = lib().fl_fedavg(layout.handle, G, _bufs(replicas, G, n, 2, "replicas"), w, fp,
                         _buf(master_out, n, 4, "master_out"),
                         _buf(working_out, n, 2, "working_out"), _stream(stream))
    _check(rc, "fl_fedavg")


def make_round_cfg(R, G, A, weights, hp, *, self_group=0, grad_scale=None, step0=1,
                   replica_fp=None, phase_events=None, step_lr=None, max_grad_norm=0.0,
                   grad_scratch=None):
    """Build an fl_round_cfg; the returned object keeps its arrays alive.
    weights and replica_fp have G entries, step_lr A, phase_events A + 2;
    grad_scratch is None or a CUDA float32 tensor of the layout's length."""
    w = _host_list([float(x) for x in weights], G, ctypes.c_float, "weights")
    fp = None if replica_fp is None else _host_list([int(x) for x in replica_fp], G,
                                                    ctypes.c_uint64, "replica_fp")
    ev = None if phase_events is None else _host_list(phase_events, A + 2, ctypes.c_void_p,
                                                      "phase_events")
    lrs = None if step_lr is None else _host_list([float(x) for x in step_lr], A, ctypes.c_float,
                                                  "step_lr")
    scratch = None if grad_scratch is None else _buf(grad_scratch, grad_scratch.numel(), 4,
                                                     "grad_scratch")
    cfg = RoundCfg(R, G, A, self_group, float(1.0 / R if grad_scale is None else grad_scale),
                   hparams(hp), int(step0), w, fp, ev, lrs, float(max_grad_norm), scratch)
    cfg._keep = (w, fp, ev, lrs, grad_scratch)
    return cfg


def _check_cfg(layout, cfg):
    """The round configuration's tensor fields against the layout."""
    keep = getattr(cfg, "_keep", None)
    scratch = keep[4] if keep is not None and len(keep) > 4 else None
    if scratch is not None:
        _buf(scratch, layout.n, 4, "grad_scratch")


def lr_cosine(t, total_steps, warmup_steps, lr_max, lr_min=0.0):
    """fl_lr_cosine: the scheduled learning rate of optimiser step t."""
    return lib().fl_lr_cosine(int(t), int(total_steps), int(warmup_steps), float(lr_max),
                              float(lr_min))


def fl_round(layout, cfg, grads, replicas, master, m, v, working, seg_sumsq=None, stream=None):
    """grads: A*R tensors (step-major); replicas: G tensors or None (entry
    self_group is ignored)."""
    n = layout.n
    _check_cfg(layout, cfg)
    rc = lib().fl_round(layout.handle, ctypes.byref(cfg),
                        _bufs(grads, cfg.A * cfg.R, n, 2, "grads"),
                        _bufs(replicas, cfg.G, n, 2, "replicas"), _buf(master, n, 4, "master"),
                        _buf(m, n, 4, "m"), _buf(v, n, 4, "v"), _buf(working, n, 2, "working"),
                        _buf(seg_sumsq, cfg.A * layout.n_seg, 4, "seg_sumsq"), _stream(stream))
    _check(rc, "fl_round")


def fl_round_noalloc(layout, cfg, grads, replicas, master, m, v, working, seg_sumsq=None,
                     stream=None):
    """fl_round with the per-segment workspace in the library's static
    scratch: allocates nothing (see include/flround.h)."""
    n = layout.n
    _check_cfg(layout, cfg)
    rc = lib().fl_round_noalloc(layout.handle, ctypes.byref(cfg),
                                _bufs(grads, cfg.A * cfg.R, n, 2, "grads"),
                                _bufs(replicas, cfg.G, n, 2, "replicas"),
                                _buf(master, n, 4, "master"), _buf(m, n, 4, "m"),
                                _buf(v, n, 4, "v"), _buf(working, n, 2, "working"),
                                _buf(seg_sumsq, cfg.A * layout.n_seg, 4, "seg_sumsq"),
                                _stream(stream))
    _check(rc, "fl_round_noalloc")


def noalloc_workspace_bytes(layout):
    """Bytes of fl_round_noalloc's static scratch the layout's workspace
    needs (FL_NOALLOC_SCRATCH_BYTES is the limit)."""
    return int(lib().fl_noalloc_workspace_bytes(layout.handle))


def fl_shard_reduce_wire(layout, peer_grads, grad_scale, wire_out, stream=None):
    n, R = layout.n, len(peer_grads)
    rc = lib().fl_shard_reduce_wire(layout.handle, R, _bufs(peer_grads, R, n, 2, "peer_grads"),
                                    float(grad_scale), _buf(wire_out, n, 2, "wire_out"),
                                    _stream(stream))
    _check(rc, "fl_shard_reduce_wire")


def fl_broadcast_recv(layout, recv_master, master, working, stream=None):
    n = layout.n
    rc = lib().fl_broadcast_recv(layout.handle, _buf(recv_master, n, 4, "recv_master"),
                                 _buf(master, n, 4, "master"), _buf(working, n, 2, "working"),
                                 _stream(stream))
    _check(rc, "fl_broadcast_recv")


def make_hsdp_cfg(H, replica=0, hsdp_scale=None, fedavg_member=True):
    return HsdpCfg(int(H), int(replica), float(1.0 / H if hsdp_scale is None else hsdp_scale),
                   1 if fedavg_member else 0)


def fl_round_hsdp(layout, cfg, hcfg, grads, replica_wires, wire, replicas, bcast_master, master,
                  m, v, working, seg_sumsq=None, stream=None):
    """grads: A*R tensors; replica_wires: A*H tensors or None (entry
    a*H + replica ignored), or None when H == 1; wire: bf16 scratch (H > 1);
    replicas: G tensors/None (FedAvg member) or None; bcast_master: fp32
    tensor (non-member) or None."""
    n = layout.n
    _check_cfg(layout, cfg)
    rc = lib().fl_round_hsdp(
        layout.handle, ctypes.byref(cfg), ctypes.byref(hcfg),
        _bufs(grads, cfg.A * cfg.R, n, 2, "grads"),
        None if replica_wires is None else _bufs(replica_wires, cfg.A * hcfg.H, n, 2,
                                                 "replica_wires"),
        _buf(wire, n, 2, "wire"),
        None if replicas is None else _bufs(replicas, cfg.G, n, 2, "replicas"),
        _buf(bcast_master, n, 4, "bcast_master"), _buf(master, n, 4, "master"),
        _buf(m, n, 4, "m"), _buf(v, n, 4, "v"), _buf(working, n, 2, "working"),
        _buf(seg_sumsq, cfg.A * layout.n_seg, 4, "seg_sumsq"), _stream(stream))
    _check(rc, "fl_round_hsdp")


def fl_grad_sumsq(layout, peer_grads, grad_scale, total_sumsq, seg_sumsq=None, stream=None):
    """total_sumsq: a CUDA float64 tensor of one element."""
    n, R = layout.n, len(peer_grads)
    rc = lib().fl_grad_sumsq(layout.handle, R, _bufs(peer_grads, R, n, 2, "peer_grads"),
                             float(grad_scale), _buf(total_sumsq, 1, 8, "total_sumsq"),
                             _buf(seg_sumsq, layout.n_seg, 4, "seg_sumsq"), _stream(stream))
    _check(rc, "fl_grad_sumsq")


def fl_local_step_clipped(layout, hp, step, peer_grads, grad_scale, total_sumsq, max_norm, master,
                          m, v, working, stream=None):
    h = hparams(hp)
    n, R = layout.n, len(peer_grads)
    rc = lib().fl_local_step_clipped(layout.handle, ctypes.byref(h), int(step), R,
                                     _bufs(peer_grads, R, n, 2, "peer_grads"), float(grad_scale),
                                     _buf(total_sumsq, 1, 8, "total_sumsq"), float(max_norm),
                                     _buf(master, n, 4, "master"), _buf(m, n, 4, "m"),
                                     _buf(v, n, 4, "v"), _buf(working, n, 2, "working"),
                                     _stream(stream))
    _check(rc, "fl_local_step_clipped")


def fl_fedopt(layout, replicas, weights, outer, prev, buf, master_out, working_out,
              replica_fp=None, stream=None):
    n, G = layout.n, len(replicas)
    w = _host_list([float(x) for x in weights], G, ctypes.c_float, "weights")
    fp = None if replica_fp is None else _host_list([int(x) for x in replica_fp], G,
                                                    ctypes.c_uint64, "replica_fp")
    o = outer_hparams(outer)
    rc = lib().fl_fedopt(layout.handle, G, _bufs(replicas, G, n, 2, "replicas"), w, fp,
                         ctypes.byref(o), _buf(prev, n, 4, "prev"), _buf(buf, n, 4, "buf"),
                         _buf(master_out, n, 4, "master_out"),
                         _buf(working_out, n, 2, "working_out"), _stream(stream))
    _check(rc, "fl_fedopt")


def fl_round_outer(layout, cfg, outer, grads, replicas, prev, buf, master, m, v, working,
                   seg_sumsq=None, stream=None):
    o = outer_hparams(outer)
    n = layout.n
    _check_cfg(layout, cfg)
    rc = lib().fl_round_outer(layout.handle, ctypes.byref(cfg), ctypes.byref(o),
                              _bufs(grads, cfg.A * cfg.R, n, 2, "grads"),
                              _bufs(replicas, cfg.G, n, 2, "replicas"), _buf(prev, n, 4, "prev"),
                              _buf(buf, n, 4, "buf"), _buf(master, n, 4, "master"),
                              _buf(m, n, 4, "m"), _buf(v, n, 4, "v"),
                              _buf(working, n, 2, "working"),
                              _buf(seg_sumsq, cfg.A * layout.n_seg, 4, "seg_sumsq"),
                              _stream(stream))
    _check(rc, "fl_round_outer")


# ---- HIP events (for fl_round's per-phase timing) -------------------------

_hip = None


def hip_runtime():
    global _hip
    if _hip is None:
        h = None
        for name in ("libamdhip64.so", "libamdhip64.so.7", "/opt/rocm/lib/libamdhip64.so"):
            try:
                h = ctypes.CDLL(name)
                break
            except OSError:
                continue
        if h is None:
            raise RuntimeError("HIP runtime library not found")
        h.hipMalloc.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t]
        h.hipFree.argtypes = [ctypes.c_void_p]
        h.hipGetDevice.argtypes = [ctypes.POINTER(ctypes.c_int)]
        h.hipSetDevice.argtypes = [ctypes.c_int]
        h.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        h.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        h.hipEventDestroy.argtypes = [ctypes.c_void_p]
        h.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        h.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                          ctypes.c_void_p]
        _hip = h
    return _hip


# hipEventCreateWithFlags flag: no system-scope fence (cache write-back and
# invalidation) when the event is recorded; for events that only time work.
HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000


class HipEvents:
    """k raw hipEvent_t handles, for fl_round's phase_events (created with
    hipEventCreateWithFlags(flags))."""

    def __init__(self, k, flags=0):
        h = hip_runtime()
        self.handles = []
        for _ in range(k):
            e = ctypes.c_void_p()
            if h.hipEventCreateWithFlags(ctypes.byref(e), ctypes.c_uint(flags)) != 0:
                raise RuntimeError("hipEventCreateWithFlags failed")
            self.handles.append(e.value)

    def elapsed_ms(self, i, j):
        h = hip_runtime()
        out = ctypes.c_float()
        if h.hipEventElapsedTime(ctypes.byref(out), self.handles[i], self.handles[j]) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return out.value

    def record(self, i, stream):
        if hip_runtime().hipEventRecord(self.handles[i], stream) != 0:
            raise RuntimeError("hipEventRecord failed")

    def synchronize(self, i):
        if hip_runtime().hipEventSynchronize(self.handles[i]) != 0:
            raise RuntimeError("hipEventSynchronize failed")

    def close(self):
        h = hip_runtime()
        for e in self.handles:
            h.hipEventDestroy(e)
        self.handles = []
