"""The synthetic workloads of the parameter-sync path.

Each workload fixes one GPU's flat shard (length N, split into segments that
carry a weight-decay flag), the round shape (R peers, G federation groups,
A local steps), the FedAvg weights, the AdamW hyperparameters and the
generator specs of every input array.  Sizes and distributions follow the
method's setting: Llama-3.1-8B trained in bf16 with AdamW at lr 3e-4 and an
aggregation every 8 local steps (Section 5, experimental setup), sharded
FSDP-style, each layer cut into S equal slices, one per GPU of a sharding
group (Section 2, FSDP).

Stream ids: master 1; gradient array k -> 1000 + k; drift of group g ->
2000 + g; layout and weight draws 3000..3009.
"""
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from . import (DRIFT_BF16, DRIFT_F32, NORMAL_BF16, NORMAL_F32, STUDENT3_BF16, host_draws,
               spec)

ADAMW = dict(lr=3e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)

MASTER_STREAM = 1
GRAD_STREAM0 = 1000
DRIFT_STREAM0 = 2000
LAYOUT_STREAM = 3000
WIRE_STREAM0 = 4000
BCAST_STREAM = 2500

MASTER_STD = 0.02
GRAD_STD = 1e-3
DRIFT_STD = 1e-4

# Llama-3.1-8B (public architecture): vocabulary 128256, hidden 4096,
# 32 decoder layers, MLP width 14336, 8 KV heads of 128.
LLAMA31_8B = dict(vocab=128256, hidden=4096, layers=32, mlp=14336, kv=1024)


def llama31_8b_segments(S):
    """Flat shard of one rank in an S-way sharding group: each parameter's
    dim-0 slice of 1/S, in module order embed; 32 x [q, k, v, o, gate, up,
    down, input_norm, post_attn_norm]; lm_head.  Returns (sizes, decay)
    where decay is 1 for 2-D weights and 0 for the norm vectors."""
    c = LLAMA31_8B
    h = c["hidden"]
    mats = [
        (c["vocab"], h),  # embed
    ]
    per_layer = [(h, h), (c["kv"], h), (c["kv"], h), (h, h), (c["mlp"], h), (c["mlp"], h),
                 (h, c["mlp"]), (h,), (h,)]
    shapes = list(mats)
    for _ in range(c["layers"]):
        shapes.extend(per_layer)
    shapes.append((c["vocab"], h))  # lm_head
    sizes, decay = [], []
    for shp in shapes:
        if shp[0] % S:
            raise ValueError("dim 0 of %r does not divide by S=%d" % (shp, S))
        rows = shp[0] // S
        sizes.append(rows * (shp[1] if len(shp) == 2 else 1))
        decay.append(1 if len(shp) == 2 else 0)
    return np.array(sizes, dtype=np.int64), np.array(decay, dtype=np.uint8)


def offsets_from_sizes(sizes):
    off = np.zeros(len(sizes) + 1, dtype=np.int64)
    np.cumsum(np.asarray(sizes, dtype=np.int64), out=off[1:])
    return off


def _uniform_ints(seed, stream, sub, n, lo, hi):
    """n integers uniform in [lo, hi] from the counter-based draws."""
    d = host_draws(seed, stream, sub, 0, n)
    span = np.uint64(hi - lo + 1)
    return (d % span).astype(np.int64) + lo


def stress_segments(seed=0, n_seg=1000, max_size=131071):
    """n_seg sizes uniform in 1..max_size, a size that is a multiple of 256
    redrawn (from the next draw index), and a 2-D flag Bernoulli(1/2)."""
    sizes = []
    j = 0
    d = host_draws(seed, LAYOUT_STREAM, 0, 0, 4 * n_seg)
    while len(sizes) < n_seg:
        s = int(d[j] % np.uint64(max_size)) + 1
        j += 1
        if s % 256:
            sizes.append(s)
    flags = (host_draws(seed, LAYOUT_STREAM + 1, 0, 0, n_seg) >> np.uint64(63)).astype(np.uint8)
    return np.array(sizes, dtype=np.int64), flags


@dataclass
class Workload:
    name: str
    seg_offsets: np.ndarray          # int64, n_seg + 1, [0] = 0, [-1] = n
    seg_decay: np.ndarray            # uint8, n_seg
    R: int
    G: int
    A: int
    weights: np.ndarray              # float32, G (un-normalised; the library normalises)
    master_spec: object
    grad_specs: list                 # distinct gradient arrays
    grad_index: List[int]            # A*R entries, step-major: grad_specs index
    replica_specs: list              # G entries; None at self_group
    working_spec: object             # initial working copy
    hp: dict = field(default_factory=lambda: dict(ADAMW))
    self_group: int = 0
    step0: int = 1
    grad_scale: Optional[float] = None
    note: str = ""
    # FL+HSDP: H replicas of the sharding group; this rank is `replica`;
    # hsdp_member: it joins FedAvg (else it receives the broadcast)
    H: int = 1
    replica: int = 0
    hsdp_member: bool = True
    wire_specs: list = field(default_factory=list)   # A*H entries, None at own index
    bcast_spec: object = None
    # outer optimiser (None: plain FedAvg): dict(lr, momentum, nesterov); the
    # outer state starts at prev = the initial master, buf = 0
    outer: Optional[dict] = None
    # global-norm clipping of each local step's gradient (0: off); with
    # clip_scratch the round gets an N-float scratch for the reduced gradient
    max_grad_norm: float = 0.0
    clip_scratch: bool = False

    def __post_init__(self):
        if self.grad_scale is None:
            self.grad_scale = 1.0 / self.R
        assert len(self.grad_index) == self.A * self.R
        assert len(self.replica_specs) == self.G
        assert self.replica_specs[self.self_group] is None

    @property
    def n(self):
        return int(self.seg_offsets[-1])

    @property
    def n_seg(self):
        return len(self.seg_offsets) - 1

    def step_bytes_per_param(self):
        """Algorithmic HBM bytes per parameter of one local step: R bf16
        gradients read, fp32 master/m/v read and written, bf16 working copy
        written; with H > 1 replicas also the own bf16 wire shard written and
        the H wire shards read."""
        base = 2 * self.R + 12 + 12 + 2
        if self.H > 1:
            base += 2 + 2 * self.H
        if self.max_grad_norm > 0:
            base += 2 * (self.H if self.H > 1 else self.R)   # the sum-of-squares pass
            if self.H == 1 and self.clip_scratch:
                # the first pass also writes the reduced gradient (4) and the
                # step reads it back (4) instead of the R peer gradients
                base += 8 - 2 * self.R
        return base

    def fedavg_bytes_per_param(self):
        """G bf16 replicas read (own working copy included), fp32 master and
        bf16 working copy written; a broadcast receiver reads the fp32 shard
        instead."""
        if self.H > 1 and not self.hsdp_member:
            return 4 + 4 + 2
        if self.outer is not None:
            return 2 * self.G + 4 + 2 + 16   # + prev and buf read and written
        return 2 * self.G + 4 + 2

    def round_bytes(self):
        return self.n * (self.A * self.step_bytes_per_param() + self.fedavg_bytes_per_param())

    def span_layout(self, lo, hi):
        """The segments of elements lo..hi-1 as a layout of their own:
        (offsets relative to lo, decay flags, index of the first segment)."""
        inner = self.seg_offsets[(self.seg_offsets > lo) & (self.seg_offsets < hi)]
        off = np.concatenate([[lo], inner, [hi]]).astype(np.int64) - lo
        first = int(np.searchsorted(self.seg_offsets, lo, side="right")) - 1
        return off, self.seg_decay[first:first + off.size - 1].copy(), first

    def describe(self):
        d = dict(workload=self.name, n=self.n, n_seg=self.n_seg, R=self.R, G=self.G,
                 A=self.A, distinct_grad_arrays=len(self.grad_specs))
        if self.H > 1:
            d.update(H=self.H, replica=self.replica, fedavg_member=self.hsdp_member)
        if self.outer is not None:
            d.update(outer=self.outer)
        if self.max_grad_norm > 0:
            d.update(max_grad_norm=self.max_grad_norm)
        return d


def _replicas(G, self_group, seed, mean=0.0, std=MASTER_STD, drift=DRIFT_STD):
    reps = []
    for g in range(G):
        if g == self_group:
            reps.append(None)
        else:
            reps.append(spec(DRIFT_BF16, MASTER_STREAM, seed, mean, std,
                             stream2=DRIFT_STREAM0 + g, std2=drift))
    return reps


def _normal_grads(n_arrays, seed, std=GRAD_STD):
    return [spec(NORMAL_BF16, GRAD_STREAM0 + k, seed, 0.0, std) for k in range(n_arrays)]


def make_workload(name, seg_sizes, seg_decay, R, G, A, *, weights=None, seed=0,
                  distinct_grads=True, student=False, own_drift=False, hp=None,
                  self_group=0, step0=1, grad_scale=None, note="", H=1, replica=0,
                  hsdp_member=True, outer=None, max_grad_norm=0.0, clip_scratch=False):
    """General constructor used by the named workloads and by the tests.

    distinct_grads: A*R distinct gradient arrays (else R arrays reused by
    every step).  student: gradients 1e-3 * Student-t(3) with 5 % exact
    zeros (else N(0, 1e-3)).  own_drift: the own fp32 master starts at
    base + drift_self (else at base)."""
    off = offsets_from_sizes(seg_sizes)
    n_arr = A * R if distinct_grads else R
    if student:
        grads = [spec(STUDENT3_BF16, GRAD_STREAM0 + k, seed, 0.0, GRAD_STD, p_zero=0.05)
                 for k in range(n_arr)]
    else:
        grads = _normal_grads(n_arr, seed)
    gidx = [a * R + r if distinct_grads else r for a in range(A) for r in range(R)]
    if own_drift:
        master = spec(DRIFT_F32, MASTER_STREAM, seed, 0.0, MASTER_STD,
                      stream2=DRIFT_STREAM0 + self_group, std2=DRIFT_STD)
        working = spec(DRIFT_BF16, MASTER_STREAM, seed, 0.0, MASTER_STD,
                       stream2=DRIFT_STREAM0 + self_group, std2=DRIFT_STD)
    else:
        master = spec(NORMAL_F32, MASTER_STREAM, seed, 0.0, MASTER_STD)
        working = spec(NORMAL_BF16, MASTER_STREAM, seed, 0.0, MASTER_STD)
    if weights is None:
        weights = np.full(G, 1.0 / G, dtype=np.float32)
    wires = []
    bcast = None
    if H > 1:
        # the other replicas' tier-1 shards: the mean of R peers' N(0, 1e-3)
        # (reused by every step when the gradient arrays are)
        wires = [None if k == replica else
                 spec(NORMAL_BF16, WIRE_STREAM0 + (a * H if distinct_grads else 0) + k, seed, 0.0,
                      GRAD_STD / np.sqrt(R))
                 for a in range(A) for k in range(H)]
        bcast = spec(DRIFT_F32, MASTER_STREAM, seed, 0.0, MASTER_STD, stream2=BCAST_STREAM,
                     std2=DRIFT_STD)
    return Workload(name=name, seg_offsets=off, seg_decay=np.asarray(seg_decay, np.uint8),
                    R=R, G=G, A=A, weights=np.asarray(weights, np.float32), master_spec=master,
                    grad_specs=grads, grad_index=gidx,
                    replica_specs=_replicas(G, self_group, seed), working_spec=working,
                    hp=dict(hp or ADAMW), self_group=self_group, step0=step0,
                    grad_scale=grad_scale, note=note, H=H, replica=replica,
                    hsdp_member=hsdp_member, wire_specs=wires, bcast_spec=bcast,
                    outer=None if outer is None else dict(outer),
                    max_grad_norm=float(max_grad_norm), clip_scratch=bool(clip_scratch))


def tiny(seed=0):
    """1,048,576-parameter flat shard, R=4, G=2 (weights 0.5/0.5), A=4."""
    return make_workload("tiny_n1m_r4_g2_a4", [1 << 20], [1], R=4, G=2, A=4,
                         weights=[0.5, 0.5], seed=seed, distinct_grads=True)


def llama8b_s8(seed=0):
    """Llama-3.1-8B shard at sharding-group size 8: N = 1,003,782,144 in 290
    segments; R=8 peer gradients (reused by the 8 local steps); G=4 equal
    weights; A=8 (the aggregation period of Section 5)."""
    sizes, dec = llama31_8b_segments(8)
    return make_workload("llama31_8b_fsdp_s8_r8_g4_a8", sizes, dec, R=8, G=4, A=8, seed=seed,
                         distinct_grads=False)


def fedavg_heavy(seed=0):
    """250M-parameter flat shard, G=8 replicas (base + per-group drift),
    weights proportional to per-group sample counts uniform in 1..16, R=4,
    A=1."""
    counts = _uniform_ints(seed, LAYOUT_STREAM + 2, 0, 8, 1, 16).astype(np.float32)
    return make_workload("fedavg_heavy_n250m_r4_g8_a1", [250_000_000], [1], R=4, G=8, A=1,
                         weights=counts, seed=seed, distinct_grads=True, own_drift=True)


def hsdp_s4(seed=0):
    """Llama-3.1-8B shard at shard factor 4 (FL+HSDP-shaped): N =
    2,007,564,288 in 290 segments; R=4 (reused by the 8 steps); G=4 equal
    weights; A=8."""
    sizes, dec = llama31_8b_segments(4)
    return make_workload("llama31_8b_hsdp_s4_r4_g4_a8", sizes, dec, R=4, G=4, A=8, seed=seed,
                         distinct_grads=False)


def stress(seed=0):
    """1,000 odd-sized segments (sizes uniform 1..131071, no multiple of 256),
    weight decay on the segments flagged 2-D; G=16 weights uniform (0,1)
    normalised to sum 1; R=16 Student-t(3) gradients scaled 1e-3 with 5 %
    exact zeros; A=4 with distinct gradients per step."""
    sizes, flags = stress_segments(seed)
    u = (host_draws(seed, LAYOUT_STREAM + 3, 0, 0, 16) >> np.uint64(11)).astype(np.float64)
    u = (u + 1.0) / 9007199254740992.0
    w = (u / u.sum()).astype(np.float32)
    return make_workload("stress_1000seg_r16_g16_a4", sizes, flags, R=16, G=16, A=4, weights=w,
                         seed=seed, distinct_grads=True, student=True)


def hsdp_s4_h2(seed=0, member=True):
    """The FL+HSDP-shaped shard (S = 4) with its replication group made
    explicit: H = 2 replicas, two-tier gradient average, this replica the
    group's FedAvg member (member=False: the broadcast receiver)."""
    sizes, dec = llama31_8b_segments(4)
    return make_workload("llama31_8b_flhsdp_s4_h2_r4_g4_a8" + ("" if member else "_recv"), sizes,
                         dec, R=4, G=4, A=8, seed=seed, distinct_grads=False, H=2, replica=0,
                         hsdp_member=member)


DILOCO_OUTER = dict(lr=0.7, momentum=0.9, nesterov=True)


def llama8b_s8_outer(seed=0):
    """The Llama-3.1-8B S=8 round with the outer Nesterov-momentum step
    (outer lr 0.7, momentum 0.9, as DiLoCo uses) in place of plain FedAvg."""
    sizes, dec = llama31_8b_segments(8)
    return make_workload("llama31_8b_fsdp_s8_r8_g4_a8_fedmom", sizes, dec, R=8, G=4, A=8,
                         seed=seed, distinct_grads=False, outer=DILOCO_OUTER)


def llama8b_s8_clip(seed=0):
    """The Llama-3.1-8B S=8 round with every local step's gradient clipped to
    global norm 1.0: a pass that sums the squares of the reduced gradient and
    stores it in an N-float scratch, then the AdamW pass over it."""
    sizes, dec = llama31_8b_segments(8)
    return make_workload("llama31_8b_fsdp_s8_r8_g4_a8_clip1", sizes, dec, R=8, G=4, A=8,
                         seed=seed, distinct_grads=False, max_grad_norm=1.0, clip_scratch=True)


def llama8b_s8_clip_noscratch(seed=0):
    """The clipped Llama-3.1-8B S=8 round without the gradient scratch: a
    sum-of-squares pass over the R peer gradients, then the fused step
    scaled by the clip coefficient (the peer gradients are read twice)."""
    sizes, dec = llama31_8b_segments(8)
    return make_workload("llama31_8b_fsdp_s8_r8_g4_a8_clip1_noscratch", sizes, dec, R=8, G=4,
                         A=8, seed=seed, distinct_grads=False, max_grad_norm=1.0,
                         clip_scratch=False)


ALL = dict(tiny=tiny, llama8b_s8=llama8b_s8, fedavg_heavy=fedavg_heavy, hsdp_s4=hsdp_s4,
           stress=stress, hsdp_s4_h2=hsdp_s4_h2,
           hsdp_s4_h2_recv=lambda seed=0: hsdp_s4_h2(seed, member=False),
           llama8b_s8_outer=llama8b_s8_outer, llama8b_s8_clip=llama8b_s8_clip,
           llama8b_s8_clip_noscratch=llama8b_s8_clip_noscratch)


def sample_indices(w, n_random=1 << 16, seed=1, full_segments=4, max_full=4096):
    """Sorted unique element indices for sampled parity at full size: both
    ends of every segment and their neighbours, the last 64 elements, every
    element of up to `full_segments` short segments (<= max_full elements),
    and n_random uniform draws.  Returns (idx, full_seg_ids)."""
    n = w.n
    off = w.seg_offsets
    parts = []
    if n == 0:
        return np.zeros(0, np.int64), []
    parts.append(off[:-1])
    parts.append(off[:-1] + 1)
    parts.append(off[1:] - 1)
    parts.append(off[1:] - 2)
    parts.append(np.arange(max(0, n - 64), n, dtype=np.int64))
    sizes = np.diff(off)
    short = np.nonzero(sizes <= max_full)[0][:full_segments]
    for s in short:
        parts.append(np.arange(off[s], off[s + 1], dtype=np.int64))
    if n_random:
        d = host_draws(seed, LAYOUT_STREAM + 9, 0, 0, n_random)
        parts.append((d % np.uint64(n)).astype(np.int64))
    idx = np.unique(np.concatenate(parts))
    idx = idx[(idx >= 0) & (idx < n)]
    return idx, [int(s) for s in short]
