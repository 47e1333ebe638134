"""Seeded synthetic inputs for the parameter-sync path.

This package generates inputs only.  It holds none of the method's
arithmetic: it is the one module that both the oracle side (host values at
chosen indices) and the GPU side (multi-GB fills in HBM) draw inputs from, so
that both see identical bits.

  spec(...)             -- describe one generated array (a ``synth_spec``)
  host_fill / gather    -- values on the host (numpy)
  dev_fill              -- values written into a torch CUDA tensor
  workloads             -- the synthetic workloads and their layouts
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))

NORMAL_F32 = 1
NORMAL_BF16 = 2
DRIFT_F32 = 3
DRIFT_BF16 = 4
STUDENT3_BF16 = 5

_BF16_KINDS = (NORMAL_BF16, DRIFT_BF16, STUDENT3_BF16)


class SynthSpec(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int32),
        ("pad_", ctypes.c_int32),
        ("seed", ctypes.c_uint64),
        ("stream", ctypes.c_uint64),
        ("stream2", ctypes.c_uint64),
        ("mean", ctypes.c_double),
        ("std", ctypes.c_double),
        ("std2", ctypes.c_double),
        ("p_zero", ctypes.c_double),
    ]

    @property
    def is_bf16(self):
        return self.kind in _BF16_KINDS

    def key(self):
        return (self.kind, self.seed, self.stream, self.stream2, self.mean, self.std,
                self.std2, self.p_zero)

    def __repr__(self):
        return ("SynthSpec(kind=%d, seed=%d, stream=%d, stream2=%d, mean=%g, std=%g, "
                "std2=%g, p_zero=%g)" % self.key())


def spec(kind, stream, seed=0, mean=0.0, std=1.0, stream2=0, std2=0.0, p_zero=0.0):
    return SynthSpec(kind, 0, seed, stream, stream2, mean, std, std2, p_zero)


_host = None
_dev = None


def _load(path, what):
    if not os.path.exists(path):
        raise RuntimeError("%s not built: %s is missing (run synth/build.py or "
                           "__graft_entry__.build())" % (what, path))
    return ctypes.CDLL(path)


def host_lib():
    global _host
    if _host is None:
        # SYNTH_HOST_LIB names another build of synth_host.c (the sanitizer test's)
        lib = _load(os.environ.get("SYNTH_HOST_LIB") or os.path.join(HERE, "libsynth_host.so"),
                    "host generator")
        P = ctypes.POINTER(SynthSpec)
        lib.synth_host_fill.argtypes = [P, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        lib.synth_host_fill_mt.argtypes = [P, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                                           ctypes.c_int]
        lib.synth_host_gather.argtypes = [P, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
        lib.synth_host_draws.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint32,
                                         ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        lib.synth_host_normals.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int64,
                                           ctypes.c_int64, ctypes.c_void_p]
        for f in ("synth_host_log", "synth_host_cos2pi", "synth_host_sqrt"):
            getattr(lib, f).argtypes = [ctypes.c_double]
            getattr(lib, f).restype = ctypes.c_double
        _host = lib
    return _host


def dev_lib():
    global _dev
    if _dev is None:
        lib = _load(os.path.join(HERE, "libsynth_dev.so"), "device generator")
        lib.synth_dev_fill.argtypes = [ctypes.POINTER(SynthSpec), ctypes.c_int64,
                                       ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
        _dev = lib
    return _dev


def _out_array(sp, n):
    return np.empty(n, dtype=np.uint16 if sp.is_bf16 else np.float32)


def host_threads():
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:
        return 1


def host_fill(sp, i0, n, threads=None):
    """Values at indices i0..i0+n-1 (uint16 bf16 bits, or float32)."""
    out = _out_array(sp, n)
    threads = host_threads() if threads is None else threads
    rc = host_lib().synth_host_fill_mt(ctypes.byref(sp), i0, n, out.ctypes.data, threads)
    if rc != 0:
        raise ValueError("synth_host_fill failed (%d) for %r" % (rc, sp))
    return out


def host_gather(sp, idx):
    """Values at the given indices (uint16 bf16 bits, or float32)."""
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = _out_array(sp, idx.size)
    rc = host_lib().synth_host_gather(ctypes.byref(sp), idx.ctypes.data, idx.size,
                                      out.ctypes.data)
    if rc != 0:
        raise ValueError("synth_host_gather failed (%d) for %r" % (rc, sp))
    return out


def host_draws(seed, stream, sub, i0, n):
    out = np.empty(n, dtype=np.uint64)
    rc = host_lib().synth_host_draws(seed, stream, sub, i0, n, out.ctypes.data)
    if rc != 0:
        raise ValueError("synth_host_draws failed")
    return out


def host_normals(seed, stream, i0, n):
    out = np.empty(n, dtype=np.float64)
    rc = host_lib().synth_host_normals(seed, stream, i0, n, out.ctypes.data)
    if rc != 0:
        raise ValueError("synth_host_normals failed")
    return out


def dev_fill(tensor, sp, i0=0):
    """Fill a contiguous CUDA tensor (torch.float32, or a 2-byte dtype for bf16
    kinds) with the values at indices i0..i0+numel-1, on the current stream."""
    import torch

    if not tensor.is_cuda or not tensor.is_contiguous():
        raise ValueError("dev_fill needs a contiguous CUDA tensor")
    want = 2 if sp.is_bf16 else 4
    if tensor.element_size() != want:
        raise ValueError("dev_fill: element size %d, kind %d needs %d"
                         % (tensor.element_size(), sp.kind, want))
    stream = torch.cuda.current_stream(tensor.device).cuda_stream
    rc = dev_lib().synth_dev_fill(ctypes.byref(sp), i0, tensor.numel(), tensor.data_ptr(),
                                  ctypes.c_void_p(stream))
    if rc != 0:
        raise RuntimeError("synth_dev_fill failed (%d) for %r" % (rc, sp))
    return tensor
