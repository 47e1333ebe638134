"""Input buffers of a workload, filled by the synth generator.

DeviceInputs: torch CUDA tensors filled in HBM by the device build;
HostInputs: numpy arrays from the host build, for all elements or at chosen
indices (bit-identical to the device values), or, for a contiguous span of a
multi-GB shard, from the device build copied to the host (DeviceSpanFiller);
HostView: the arrays of a HostInputs restricted to a sub-range.
"""
import numpy as np

from . import dev_fill, host_fill, host_gather
from .workloads import Workload


class DeviceInputs:
    """Every input and state array of workload w on the device, filled by
    the generator's device build.  place(n, dtypes, device) -> tensors
    chooses where the arrays live (default: one allocation each)."""

    def __init__(self, w: Workload, device="cuda:0", place=None):
        import torch

        n = w.n
        self.w = w
        f32, bf = torch.float32, torch.bfloat16
        wire_keys = []
        for sp in w.wire_specs:
            if sp is not None and sp.key() not in wire_keys:
                wire_keys.append(sp.key())
        plan = ([f32, f32, f32, bf] + [bf] * len(w.grad_specs) +
                [bf] * sum(sp is not None for sp in w.replica_specs) + [bf] * len(wire_keys) +
                ([bf] if w.H > 1 else []) + ([f32, f32] if w.outer else []) +
                ([f32] if w.bcast_spec is not None else []) +
                ([f32] if w.max_grad_norm > 0 and w.clip_scratch and w.H == 1 else []))
        if place is None:
            arrays = iter([torch.empty(n, dtype=d, device=device) for d in plan])
        else:
            arrays = iter(place(n, plan, device))
        self.master = dev_fill(next(arrays), w.master_spec)
        self.m = next(arrays).zero_()
        self.v = next(arrays).zero_()
        self.working = dev_fill(next(arrays), w.working_spec)
        self.grad_arrays = [dev_fill(next(arrays), sp) for sp in w.grad_specs]
        self.grads = [self.grad_arrays[k] for k in w.grad_index]
        self.replicas = [None if sp is None else dev_fill(next(arrays), sp)
                         for sp in w.replica_specs]
        filled = {}
        for sp in w.wire_specs:
            if sp is not None and sp.key() not in filled:
                filled[sp.key()] = dev_fill(next(arrays), sp)
        self.replica_wires = [None if sp is None else filled[sp.key()]
                              for sp in w.wire_specs] or None
        self.wire = next(arrays) if w.H > 1 else None
        self.prev = dev_fill(next(arrays), w.master_spec) if w.outer else None
        self.buf = next(arrays).zero_() if w.outer else None
        self.bcast = None if w.bcast_spec is None else dev_fill(next(arrays), w.bcast_spec)
        self.grad_scratch = (next(arrays)
                             if w.max_grad_norm > 0 and w.clip_scratch and w.H == 1 else None)
        assert next(arrays, None) is None

    def bytes(self):
        t = [self.master, self.m, self.v, self.working] + self.grad_arrays + \
            [r for r in self.replicas if r is not None] + \
            list({id(r): r for r in (self.replica_wires or []) if r is not None}.values()) + \
            [x for x in (self.wire, self.bcast, self.prev, self.buf, self.grad_scratch)
             if x is not None]
        return sum(x.numel() * x.element_size() for x in t)


def to_u16(t):
    import torch

    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def gather_u16(t, idx_dev):
    import torch

    return to_u16(torch.index_select(t.view(torch.int16), 0, idx_dev))


def gather_f32(t, idx_dev):
    import torch

    return torch.index_select(t, 0, idx_dev).cpu().numpy()


class HostInputs:
    """The same inputs on the host, for all elements or at given indices."""

    def __init__(self, w: Workload, idx=None, span=None, fill=None):
        """idx: element indices (sorted), or span: a contiguous (lo, hi)
        range; neither: the whole shard.  fill(spec) -> array overrides how
        the values of a span are produced (DeviceSpanFiller)."""
        self.w = w
        if fill is not None:
            pass
        elif span is not None:
            lo, hi = int(span[0]), int(span[1])
            fill = lambda sp: host_fill(sp, lo, hi - lo)  # noqa: E731
        elif idx is None:
            fill = lambda sp: host_fill(sp, 0, w.n)  # noqa: E731
        else:
            fill = lambda sp: host_gather(sp, idx)  # noqa: E731
        self.master = fill(w.master_spec)
        n = self.master.size
        self.m = np.zeros(n, np.float32)
        self.v = np.zeros(n, np.float32)
        self.working = fill(w.working_spec)
        # read-only inputs with the same spec share one array
        memo = {}

        def once(sp):
            if sp.key() not in memo:
                memo[sp.key()] = fill(sp)
            return memo[sp.key()]

        self.grad_arrays = [once(sp) for sp in w.grad_specs]
        self.grads = [self.grad_arrays[k] for k in w.grad_index]
        self.replicas = [None if sp is None else once(sp) for sp in w.replica_specs]
        self.replica_wires = [None if sp is None else once(sp) for sp in w.wire_specs] or None
        self.bcast = None if w.bcast_spec is None else fill(w.bcast_spec)
        self.prev = fill(w.master_spec) if w.outer else None
        self.buf = np.zeros(n, np.float32) if w.outer else None


_ARRAYS = ("master", "m", "v", "working", "prev", "buf", "bcast")
_LISTS = ("grad_arrays", "replicas", "replica_wires")


class HostView:
    """The arrays of a HostInputs restricted to elements a..b-1 (numpy views:
    writes go to the parent's arrays)."""

    def __init__(self, host, a, b):
        self.w = host.w
        for k in _ARRAYS:
            x = getattr(host, k, None)
            setattr(self, k, None if x is None else x[a:b])
        for k in _LISTS:
            xs = getattr(host, k, None)
            setattr(self, k, None if xs is None else [None if x is None else x[a:b] for x in xs])
        self.grads = [self.grad_arrays[k] for k in self.w.grad_index]


class DeviceSpanFiller:
    """Values of a contiguous span produced by the generator's device build
    (synth_dev) into one scratch tensor and copied to the host: the same bits
    as the host build (both builds evaluate one source), at HBM speed, for
    spans of shards too large to regenerate on the host in reasonable time.
    It touches no buffer of the library under test.  check(spec, lo, values)
    compares `n_check` random elements of each span with the host build."""

    def __init__(self, max_span, n_check=2048, device="cuda:0"):
        import torch

        self.torch = torch
        self.scratch = torch.empty(max_span, dtype=torch.float32, device=device)
        self.n_check = n_check
        self.rng = np.random.default_rng(12345)
        self.checked = 0

    def fill(self, sp, lo, hi):
        torch = self.torch
        n = hi - lo
        if n > self.scratch.numel():
            raise ValueError("span longer than the scratch tensor")
        if sp.is_bf16:
            t = self.scratch.view(torch.int16)[:n]
        else:
            t = self.scratch[:n]
        dev_fill(t, sp, i0=lo)
        out = t.cpu().numpy()
        out = out.view(np.uint16) if sp.is_bf16 else out
        if self.n_check and n:
            k = min(self.n_check, n)
            j = np.sort(self.rng.choice(n, size=k, replace=False))
            ref = host_gather(sp, j.astype(np.int64) + lo)
            if not np.array_equal(out[j].view(ref.dtype), ref):
                raise AssertionError("device generator differs from the host build on %r" % sp)
            self.checked += k
        return out

    def host_inputs(self, w, lo, hi):
        """A HostInputs of elements lo..hi-1 filled through the device build."""
        return HostInputs(w, span=(lo, hi), fill=lambda sp: self.fill(sp, lo, hi))
