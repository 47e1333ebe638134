"""The C ABI without a GPU: the library loads, exports every symbol the
header declares, and its host-side logic (status strings, fingerprints,
argument validation that happens before any HIP call) behaves."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2609_20359_amd as P
from paper_2609_20359_amd import flround as F

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "flround.h")


def header_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(fl_[a-z0-9_]+)\s*\(", src)))


def test_header_declares_the_binding_exports():
    assert header_functions() == sorted(F.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(F.LIB_PATH)
    missing = [f for f in header_functions() if not hasattr(lib, f)]
    assert not missing, missing


def test_status_strings_and_version():
    assert P.status_string(0) == "FL_OK"
    for code in range(-7, 0):
        assert P.status_string(code).startswith("FL_ERR_")
    assert "unknown" in P.status_string(7)
    assert P.lib().fl_version() >> 16 == 1
    assert P.lib().fl_version() & 0xFFFF >= 7   # NULL phase_events entries


def test_fingerprint_host():
    off = np.array([0, 512, 4096, 10000], np.int64)
    dec = np.array([1, 0, 1], np.uint8)
    a = P.fingerprint(off, dec)
    assert a != 0
    assert a == P.fingerprint(off.copy(), dec.copy())
    assert a == P.fingerprint(off, np.array([7, 0, 1], np.uint8))     # flags are 0/1
    assert a != P.fingerprint(off, np.array([1, 1, 1], np.uint8))     # decay differs
    assert a != P.fingerprint(np.array([0, 513, 4096, 10000]), dec)   # boundary differs
    assert P.fingerprint(off) == P.fingerprint(off, np.ones(3, np.uint8))
    # invalid layouts hash to 0
    L = P.lib()
    bad = np.array([0, 10, 10, 20], np.int64)
    assert L.fl_fingerprint(20, 3, bad.ctypes.data, None) == 0
    assert L.fl_fingerprint(21, 3, off.ctypes.data, None) == 0
    assert L.fl_fingerprint(-1, 0, off.ctypes.data, None) == 0


def test_layout_create_rejects_bad_layouts_without_a_gpu():
    L = P.lib()
    h = ctypes.c_void_p()
    cases = [
        (10, 2, np.array([0, 5, 5], np.int64)),      # empty segment
        (10, 2, np.array([1, 5, 10], np.int64)),     # does not start at 0
        (10, 2, np.array([0, 5, 9], np.int64)),      # does not end at n
        (10, 0, np.array([0], np.int64)),            # n > 0 needs a segment
        (-5, 1, np.array([0, -5], np.int64)),        # negative n
    ]
    for n, ns, off in cases:
        assert L.fl_layout_create(n, ns, off.ctypes.data, None, ctypes.byref(h)) == -1
    assert L.fl_layout_create(10, 1, None, None, ctypes.byref(h)) == -1
    assert L.fl_layout_create(10, 1, np.array([0, 10]).ctypes.data, None, None) == -1


def test_layout_tables_are_built_before_the_device_is_needed():
    """Valid layouts of several shapes go through the host-side table build
    (tiles, pieces, finalize chunks) and only then ask for the device: with
    no GPU the call returns FL_ERR_HIP and no handle."""
    L = P.lib()
    r = np.random.default_rng(5)
    shapes = [
        np.array([1], np.int64),                                  # one element
        np.array([2048 * 1025 + 7], np.int64),                    # a two-chunk segment
        np.ones(5000, np.int64),                                  # 5000 one-element segments
        r.integers(1, 5000, 777).astype(np.int64),                # ragged
        np.array([3, 2048 * 3, 1, 1, 2047, 2049, 5], np.int64),   # straddling tiles
    ]
    for sizes in shapes:
        off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
        dec = (np.arange(sizes.size) % 2).astype(np.uint8)
        h = ctypes.c_void_p()
        rc = L.fl_layout_create(int(off[-1]), sizes.size, off.ctypes.data, dec.ctypes.data,
                                ctypes.byref(h))
        assert rc == -5 and not h.value


def test_calls_reject_null_handles_without_a_gpu():
    L = P.lib()
    cfg = F.make_round_cfg(2, 2, 1, [1.0, 1.0], dict(lr=3e-4, beta1=0.9, beta2=0.95, eps=1e-8,
                                                   weight_decay=0.1))
    arr = (ctypes.c_void_p * 4)()
    assert L.fl_round(None, ctypes.byref(cfg), arr, arr, None, None, None, None, None, None) == -1
    assert L.fl_fedavg(None, 2, arr, None, None, None, None, None) == -1
    assert L.fl_shard_reduce(None, 1, arr, ctypes.c_float(1.0), None, None, None) == -1
    h = F.hparams(dict(lr=3e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1))
    assert L.fl_adamw_step(None, ctypes.byref(h), 1, None, None, None, None, None, None) == -1
    assert L.fl_layout_numel(None) == -1
    assert L.fl_layout_fingerprint(None) == 0
    assert L.fl_layout_destroy(None) == 0


def test_blocks_per_cu_setting_round_trips():
    prev = P.set_blocks_per_cu(5)
    assert P.set_blocks_per_cu(prev) == 5


def test_lr_cosine_matches_the_oracle_and_transformers():
    import oracle
    import transformers
    import torch

    orc = oracle.Oracle()
    for T, W, lr_max, lr_min in ((64, 7, 3e-4, 0.0), (300, 30, 1e-3, 1e-5)):
        base = float(np.float32(lr_max))
        p = torch.nn.Parameter(torch.zeros(1))
        opt = torch.optim.SGD([p], lr=base)
        if lr_min:
            sch = transformers.get_cosine_with_min_lr_schedule_with_warmup(
                opt, W, T, min_lr_rate=float(np.float32(lr_min)) / base)
        else:
            sch = transformers.get_cosine_schedule_with_warmup(opt, W, T)
        for t in range(1, T + 2):
            lib_lr = np.float32(P.lr_cosine(t, T, W, lr_max, lr_min))
            assert lib_lr == np.float32(orc.lr_cosine(t, T, W, lr_max, lr_min))
            assert lib_lr == np.float32(opt.param_groups[0]["lr"])
            opt.step()
            sch.step()


def test_binding_checks_host_lists_and_tensors_without_a_gpu():
    """The binding checks every list length and tensor on the host before it
    calls the library, so a mismatch never reaches a kernel."""
    import pytest
    import torch

    hp = dict(lr=3e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)
    with pytest.raises(ValueError):
        F.make_round_cfg(2, 3, 1, [1.0, 1.0], hp)                     # G weights
    with pytest.raises(ValueError):
        F.make_round_cfg(2, 2, 3, [1.0, 1.0], hp, step_lr=[1e-3, 1e-3])
    with pytest.raises(ValueError):
        F.make_round_cfg(2, 2, 1, [1.0, 1.0], hp, replica_fp=[1])
    with pytest.raises(ValueError):
        F.make_round_cfg(2, 2, 1, [1.0, 1.0], hp, phase_events=[0, 0])  # needs A + 2

    class FakeLayout:  # a layout needs a GPU; the checks below come first
        handle, n, n_seg = None, 16, 1

    cfg = F.make_round_cfg(2, 2, 1, [1.0, 1.0], hp)
    cpu = torch.zeros(16, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="CUDA"):
        F.fl_round(FakeLayout, cfg, [cpu, cpu], [None, cpu], None, None, None, None)
    with pytest.raises(ValueError, match="entries"):
        F.fl_round(FakeLayout, cfg, [None] * 3, [None, None], None, None, None, None)
    with pytest.raises(ValueError, match="entries"):
        F.fl_fedavg(FakeLayout, [None, None], [1.0], None, None)


def test_binding_fails_loudly_without_the_library(monkeypatch, tmp_path):
    """No fallback: with the library absent every call raises."""
    import pytest

    monkeypatch.setattr(F, "_lib", None)
    monkeypatch.setattr(F, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="not built"):
        F.lib()
    with pytest.raises(RuntimeError, match="not built"):
        F.lr_cosine(1, 10, 1, 1e-3)


def test_place_arrays_layout():
    """The staggered placement: one allocation, array k at a 2 MiB boundary
    plus k x 2 KiB, each a contiguous tensor of n elements of its dtype, no
    two overlapping (checked on host memory)."""
    import torch

    from paper_2609_20359_amd import arena

    n = 100_003
    dtypes = [torch.float32, torch.float32, torch.bfloat16] + [torch.bfloat16] * 5
    ts = arena.place_arrays(n, dtypes, device="cpu")
    assert [t.dtype for t in ts] == dtypes
    assert all(t.numel() == n and t.is_contiguous() for t in ts)
    base = ts[0].data_ptr()
    assert len({t.untyped_storage().data_ptr() for t in ts}) == 1   # one allocation
    spans = []
    for k, t in enumerate(ts):
        assert (t.data_ptr() - base) % arena.ALIGN == k * arena.STRIDE
        spans.append((t.data_ptr(), t.data_ptr() + n * t.element_size()))
    spans.sort()
    assert all(a[1] <= b[0] for a, b in zip(spans, spans[1:]))
    for t in ts:
        t.zero_()
    ts[2].fill_(1.5)
    assert all(float(t.float().abs().max()) == 0.0 for k, t in enumerate(ts) if k != 2)


def test_separate_arrays_is_device_only():
    """The exact-size placement allocates with hipMalloc; it refuses host
    tensors rather than falling back to another allocator."""
    import torch

    with pytest.raises(ValueError, match="device memory"):
        P.separate_arrays(10, [torch.float32], device="cpu")
