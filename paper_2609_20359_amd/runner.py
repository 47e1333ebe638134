"""One round of a workload through the C ABI.

A workload (synth.workloads.Workload) fixes the round shape, hyperparameters
and tensors; these helpers only turn it into the arguments of fl_round,
fl_round_hsdp or fl_round_outer (marshalling, no arithmetic).  The benchmark
and the GPU tests both use them.
"""
from . import flround as F


def round_cfg(w, step0=None, phase_events=None, dev=None, step_lr=None):
    """The fl_round_cfg of workload w (with dev: its gradient scratch, if the
    workload has one)."""
    scratch = None if dev is None else getattr(dev, "grad_scratch", None)
    return F.make_round_cfg(w.R, w.G, w.A, w.weights, w.hp, self_group=w.self_group,
                            grad_scale=w.grad_scale, step0=w.step0 if step0 is None else step0,
                            phase_events=phase_events, max_grad_norm=w.max_grad_norm,
                            grad_scratch=scratch, step_lr=step_lr)


def gpu_round(layout, w, dev, seg_sumsq=None, phase_events=None, cfg=None, stream=None):
    """One fl_round (fl_round_hsdp when w.H > 1, fl_round_outer with an outer
    step) on the device tensors of dev; returns the configuration used."""
    if cfg is None:
        cfg = round_cfg(w, phase_events=phase_events, dev=dev)
    if w.outer is not None:
        F.fl_round_outer(layout, cfg, w.outer, dev.grads, dev.replicas, dev.prev, dev.buf,
                         dev.master, dev.m, dev.v, dev.working, seg_sumsq=seg_sumsq,
                         stream=stream)
    elif w.H > 1:
        hc = F.make_hsdp_cfg(w.H, w.replica, 1.0 / w.H, w.hsdp_member)
        F.fl_round_hsdp(layout, cfg, hc, dev.grads, dev.replica_wires, dev.wire,
                        dev.replicas if w.hsdp_member else None,
                        None if w.hsdp_member else dev.bcast, dev.master, dev.m, dev.v,
                        dev.working, seg_sumsq=seg_sumsq, stream=stream)
    else:
        F.fl_round(layout, cfg, dev.grads, dev.replicas, dev.master, dev.m, dev.v, dev.working,
                   seg_sumsq=seg_sumsq, stream=stream)
    return cfg
