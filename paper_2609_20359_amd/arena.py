"""Placement of a shard's N-sized arrays in HBM.

The C ABI takes any 16-byte-aligned device pointers, so where the arrays of a
shard live is the caller's choice.  Two placements are offered to callers that
allocate a shard's arrays together:

  place_arrays()      one allocation for all, array k starting at a 2 MiB
                      boundary plus k x 2 KiB (what the benchmark and the
                      full-size tests use)
  separate_arrays()   one hipMalloc per array, of exactly the array's bytes

Why it matters: the fused step streams about a dozen arrays at the same
element index at once (the R peer gradients, master, m, v and the working
copy), and how their pages fall on HBM's channels and banks moves its rate by
up to a seventh.  Rounds of the Llama-3.1-8B shard at S = 8 (R = 8) on
MI355X, one placement per fresh process, on two kinds of box:

                                      box kind A           box kind B
  one pool, 2 KiB stagger             63.4-63.7 ms (3)     63.8-65.0 ms (11)
  one hipMalloc per array             67.2-67.5 ms (8)     58.2-63.8 ms (11)
  torch's caching allocator           67.3-67.4 ms (3)     59.1-67.0 ms (6)

On boxes of kind A separate allocations land the same way in every process;
on kind B the HIP runtime places them anew in each and the rate follows.
The staggered pool gives the same rate on both, which is why it is the
default; the same-design bandwidth probe, its streams placed either way,
shows the same spread.  Changing which workgroup walks which tiles (one
contiguous range per workgroup, or chunks of 16 or 128 tiles dealt round
robin) moved the probe's rate no more than a new placement does."""
import atexit
import ctypes

ALIGN = 2 << 20     # large allocations start on 2 MiB boundaries
STRIDE = 2 << 10    # staggered placement: array k starts STRIDE * k past its slot

_exiting = False


@atexit.register
def _at_exit():
    # blocks still alive when the interpreter ends are left to the process
    # exit rather than freed while the runtime may be shutting down
    global _exiting
    _exiting = True


class _HipBlock:
    """One hipMalloc'd block of device memory, exposed through the CUDA array
    interface.  A tensor made from it holds a reference to the block, so the
    block is freed (hipFree) when the last tensor on it is freed."""

    def __init__(self, nbytes, device_index):
        from .flround import hip_runtime

        h = hip_runtime()
        prev = ctypes.c_int()
        if h.hipGetDevice(ctypes.byref(prev)) != 0:
            raise RuntimeError("hipGetDevice failed")
        if h.hipSetDevice(device_index) != 0:
            raise RuntimeError("hipSetDevice(%d) failed" % device_index)
        p = ctypes.c_void_p()
        try:
            rc = h.hipMalloc(ctypes.byref(p), ctypes.c_size_t(nbytes))
        finally:
            h.hipSetDevice(prev.value)
        if rc != 0 or not p.value:
            raise MemoryError("hipMalloc of %d bytes on device %d failed (%d)"
                              % (nbytes, device_index, rc))
        self.ptr = p.value
        self.__cuda_array_interface__ = {"shape": (nbytes,), "typestr": "|u1",
                                         "data": (self.ptr, False), "version": 2,
                                         "strides": None}

    def __del__(self):
        if self.ptr and not _exiting:
            from .flround import hip_runtime

            hip_runtime().hipFree(ctypes.c_void_p(self.ptr))
        self.ptr = None


def separate_arrays(n, dtypes, device="cuda"):
    """One tensor of n elements for each dtype, each in a device allocation
    of its own of exactly n x element-size bytes (in the order given).  Each
    tensor keeps its allocation alive; it is freed with the tensor."""
    import torch

    dev = torch.device(device)
    if dev.type != "cuda":
        raise ValueError("separate_arrays allocates device memory; got %s" % dev)
    idx = dev.index if dev.index is not None else torch.cuda.current_device()
    out = []
    for d in dtypes:
        nbytes = n * torch.tensor([], dtype=d).element_size()
        if nbytes == 0:
            out.append(torch.empty(0, dtype=d, device=dev))
            continue
        blk = _HipBlock(nbytes, idx)
        t = torch.as_tensor(blk, device=torch.device("cuda", idx))
        if t.data_ptr() != blk.ptr or t.numel() != nbytes:
            raise RuntimeError("device array was copied instead of wrapped")
        out.append(t.view(d))
    return out


def place_arrays(n, dtypes, device="cuda"):
    """One tensor of n elements for each dtype, all carved from one
    allocation, array k at a 2 MiB boundary plus k x 2 KiB (in the order
    given).  The views keep the allocation alive; it is freed with the last
    of them."""
    import torch

    sizes = [n * torch.tensor([], dtype=d).element_size() for d in dtypes]
    slots = [((b + ALIGN - 1) // ALIGN) * ALIGN + ALIGN for b in sizes]
    pool = torch.empty(sum(slots) + ALIGN, dtype=torch.uint8, device=device)
    off = (-pool.data_ptr()) % ALIGN
    out = []
    for k, (d, b, s) in enumerate(zip(dtypes, sizes, slots)):
        o = off + (k * STRIDE) % ALIGN
        out.append(pool[o:o + b].view(d))
        off += s
    return out
