"""Placement of a shard's N-sized arrays in HBM.

The C ABI takes any 16-byte-aligned device pointers, so where the arrays of a
shard live is the caller's choice.  This is the placement the benchmark and
the full-size tests use, offered to callers that allocate a shard's arrays
together: place_arrays() carves them from one allocation, array k starting
at a 2 MiB boundary plus k x 2 KiB.

Why: allocated one by one, every large array starts on a 2 MiB boundary, so
the streams a kernel reads and writes at the same element index (the R peer
gradients, master, m, v and the working copy) sit at the same offset within
their 2 MiB pages.  On MI355X that costs the fused step of the Llama-3.1-8B
shard at S = 8 (R = 8) about 7 %: a round of 68.0 ms against 63.3-63.8 ms
with the 2 KiB stride, the same in four pools at different physical
addresses.  Of the uniform strides measured (256 B to 768 KiB) and of
per-array random offsets, the 2 KiB stride in this array order was the
best; it also gained 0.4-0.6 % on the R = 4 and R = 16 shards."""

ALIGN = 2 << 20     # large allocations start on 2 MiB boundaries
STRIDE = 2 << 10    # array k starts STRIDE * k past its slot's boundary


def place_arrays(n, dtypes, device="cuda"):
    """One tensor of n elements for each dtype, all carved from one
    allocation in the placement described above (in the order given).  The
    views keep the allocation alive; it is freed with the last of them."""
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
