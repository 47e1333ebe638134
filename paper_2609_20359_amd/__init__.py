"""MI355X-native parameter-sync path of FL+FSDP / FL+HSDP training.

One GPU's share of the method of "Accelerating Sharded Data Parallelism at
Scale with Federated Learning" (Section 4.2): the local arithmetic of the
gradient reduce-scatter, the AdamW step on the fp32 master shard, and the
FedAvg of the federation groups' replicas, as a C-ABI library (libflround.so,
include/flround.h) of hand-written gfx950 kernels.  The Python face below is a
thin ctypes binding with the same names.
"""
from .flround import (FL_MAX_GROUPS, FL_MAX_PEERS, FL_NOALLOC_SCRATCH_BYTES,
                      HIP_EVENT_DISABLE_SYSTEM_FENCE, FlError, HipEvents, Layout, fingerprint,
                      fl_adamw_step, fl_broadcast_recv, fl_fedavg, fl_fedopt, fl_grad_sumsq,
                      fl_local_step, fl_local_step_clipped, fl_round, fl_round_hsdp,
                      fl_round_noalloc, fl_round_outer, fl_shard_reduce,
                      fl_shard_reduce_wire, lib, lr_cosine, make_hsdp_cfg, make_round_cfg,
                      noalloc_workspace_bytes, set_blocks_per_cu, status_string)
from .arena import place_arrays, separate_arrays

__all__ = ["FL_MAX_GROUPS", "FL_MAX_PEERS", "FL_NOALLOC_SCRATCH_BYTES",
           "HIP_EVENT_DISABLE_SYSTEM_FENCE", "FlError", "HipEvents", "Layout", "fingerprint",
           "fl_adamw_step", "fl_broadcast_recv", "fl_fedavg", "fl_fedopt", "fl_grad_sumsq",
           "fl_local_step", "fl_local_step_clipped",
           "fl_round", "fl_round_hsdp", "fl_round_noalloc", "fl_round_outer", "fl_shard_reduce",
           "fl_shard_reduce_wire", "lib", "lr_cosine", "make_hsdp_cfg", "make_round_cfg",
           "noalloc_workspace_bytes", "place_arrays", "set_blocks_per_cu", "separate_arrays",
           "status_string"]
