"""Input buffers of a workload, filled by the synth generator.

DeviceInputs: torch CUDA tensors filled in HBM by the device build;
HostInputs: numpy arrays from the host build, for all elements or at chosen
indices (bit-identical to the device values).
"""
import numpy as np

from . import dev_fill, host_fill, host_gather
from .workloads import Workload


class DeviceInputs:
    def __init__(self, w: Workload, device="cuda:0"):
        import torch

        n = w.n
        self.w = w
        f32 = dict(dtype=torch.float32, device=device)
        bf = dict(dtype=torch.bfloat16, device=device)
        self.master = dev_fill(torch.empty(n, **f32), w.master_spec)
        self.m = torch.zeros(n, **f32)
        self.v = torch.zeros(n, **f32)
        self.working = dev_fill(torch.empty(n, **bf), w.working_spec)
        self.grad_arrays = [dev_fill(torch.empty(n, **bf), sp) for sp in w.grad_specs]
        self.grads = [self.grad_arrays[k] for k in w.grad_index]
        self.replicas = [None if sp is None else dev_fill(torch.empty(n, **bf), sp)
                         for sp in w.replica_specs]
        filled = {}

        def wire_buf(sp):
            if sp.key() not in filled:
                filled[sp.key()] = dev_fill(torch.empty(n, **bf), sp)
            return filled[sp.key()]

        self.replica_wires = [None if sp is None else wire_buf(sp) for sp in w.wire_specs] or None
        self.wire = torch.empty(n, **bf) if w.H > 1 else None
        self.prev = dev_fill(torch.empty(n, **f32), w.master_spec) if w.outer else None
        self.buf = torch.zeros(n, **f32) if w.outer else None
        self.bcast = None if w.bcast_spec is None else dev_fill(torch.empty(n, **f32),
                                                                 w.bcast_spec)
        self.grad_scratch = (torch.empty(n, **f32)
                             if w.max_grad_norm > 0 and w.clip_scratch and w.H == 1 else None)

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

    def __init__(self, w: Workload, idx=None, span=None):
        """idx: element indices (sorted), or span: a contiguous (lo, hi)
        range; neither: the whole shard."""
        self.w = w
        if span is not None:
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
        self.grad_arrays = [fill(sp) for sp in w.grad_specs]
        self.grads = [self.grad_arrays[k] for k in w.grad_index]
        self.replicas = [None if sp is None else fill(sp) for sp in w.replica_specs]
        self.replica_wires = [None if sp is None else fill(sp) for sp in w.wire_specs] or None
        self.bcast = None if w.bcast_spec is None else fill(w.bcast_spec)
        self.prev = fill(w.master_spec) if w.outer else None
        self.buf = np.zeros(n, np.float32) if w.outer else None
