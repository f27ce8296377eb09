"""The C-ABI library loads and exports every function include/octo.h declares; host-side
argument checks answer without a GPU."""
import ctypes
import os
import re

import pytest

from paper_2509_23722_amd import _lib, inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "octo.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return re.findall(r"^\s*(?:const\s+)?[A-Za-z_0-9]+\**\s+\**(octo_[a-z_0-9]+)\s*\(", src,
                      flags=re.M)


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert {"octo_sim_batch", "octo_tune_step", "octo_strerror"} <= set(names)
    L = ctypes.CDLL(_lib.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n


def test_record_layout_matches_inputs():
    for P, v, mp in [(1, 1, 0), (4, 1, 0), (8, 2, 0), (16, 2, 2), (32, 2, 0), (8, 8, 5), (64, 1, 0)]:
        assert _lib.record_stride(P, v, mp) == inputs.record_stride(P, v, mp)
        assert _lib.lib().octo_record_pert_offset(P, v) == inputs.pert_offset(P, v)
    assert _lib.record_stride(65, 1, 0) < 0 and _lib.record_stride(16, 8, 0) < 0


def test_argument_checks_without_gpu():
    L = _lib.lib()
    good = _lib.problem(16, 4, 1, 8, inputs.record_stride(4, 1, 0), 0)
    assert _lib.chain_stride(good) == (good.cand_stride + 24 + 16 * 4 + 15) // 16 * 16
    assert _lib.queue_capacity(good) == 3 * 1 * 8
    # rows hold a multiple of eight entries (16-byte spans)
    assert _lib.queue_capacity(_lib.problem(9, 4, 1, 5, inputs.record_stride(4, 1, 0), 0)) == 16
    bad = [
        _lib.problem(16, 65, 1, 8, 256, 0),       # P > 64
        _lib.problem(0, 4, 1, 8, 32, 0),          # L < 1
        _lib.problem(16, 4, 1, 0, 32, 0),         # M < 1
        _lib.problem(16, 4, 1, 2048, 32, 0),      # M too large
        _lib.problem(16, 4, 1, 8, 8, 0),          # stride too small
        _lib.problem(16, 4, 1, 8, 40, 0),         # stride not a multiple of 16
        _lib.problem(300, 4, 1, 8, 32, 0),        # L > 255
        _lib.problem(16, 16, 8, 8, 512, 0),       # P * v_max > 64
    ]
    for p in bad:
        assert L.octo_sim_batch(ctypes.byref(p), None, None, None, 1, None, None, None) == -1
        assert L.octo_tune_step(ctypes.byref(p), None, None, None, None, 1, 0, 0, None) == -1
        assert L.octo_tune_step_mem(ctypes.byref(p), None, None, None, 0, None, None, None, 1, 0,
                                    0, None) == -1
        assert L.octo_advance_w(ctypes.byref(p), None, None, None, None, None, 1, None, None,
                                None, None, None) == -1
        assert L.octo_alg1_tune(ctypes.byref(p), None, None, None, 1, 1, None, None, None,
                                None) == -1
    # valid problem but null arrays / negative sizes are rejected before any launch
    assert L.octo_sim_batch(ctypes.byref(good), None, None, None, 4, None, None, None) == -1
    assert L.octo_sim_batch(ctypes.byref(good), None, None, None, -1, None, None, None) == -1
    assert L.octo_alg1_tune(ctypes.byref(good), None, None, None, 4, 1, None, None, None,
                            None) == -1
    assert L.octo_alg1_tune(ctypes.byref(good), None, None, None, 4, -1, None, None, None,
                            None) == -1
    # the neighbour batch of one iteration (n x the largest neighbourhood) must fit int32
    nbig = (2**31 - 1) // (3 * 1 * 8 + 2) + 1
    assert L.octo_alg1_tune(ctypes.byref(good), None, None, None, nbig, 1, None, None, None,
                            None) == -1
    assert L.octo_tune_step(ctypes.byref(good), None, None, None, None, 2, 0, -1, None) == -1
    assert L.octo_tune_step_mem(ctypes.byref(good), None, None, None, 8, None, None, None, 2, 0,
                                0, None) == -1
    assert L.octo_tune_step_mem(ctypes.byref(good), None, None, None, 5000, None, None, None, 2,
                                0, 0, None) == -1  # max_advance above OCTO_MAX_ADVANCE
    assert L.octo_advance_w(ctypes.byref(good), None, None, None, None, None, 3, None, None, None,
                            None, None) == -1
    assert L.octo_advance_w(ctypes.byref(good), None, None, None, None, None, 0, None, None, None,
                            None, None) == 0
    # an empty batch is a no-op
    assert L.octo_sim_batch(ctypes.byref(good), None, None, None, 0, None, None, None) == 0
    assert L.octo_strerror(-1) == b"invalid argument"


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "absent.so"))
    monkeypatch.setattr(_lib, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        _lib.lib()
