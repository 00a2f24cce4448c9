"""The C-ABI library loads and exports every entry point that include/tsid.h
declares; host-only logic runs without a GPU (CPU)."""
import ctypes
import os
import re

import numpy as np

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "tsid.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tsid_[a-z_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = _declared()
    for want in ("tsid_build_template", "tsid_fit_template", "tsid_extend_chunk", "tsid_loss",
                 "tsid_create", "tsid_destroy", "tsid_sync", "tsid_export_index"):
        assert want in names


def test_library_exports_every_declared_symbol():
    from paper_2608_00977_amd import LIB_PATH, lib
    assert os.path.exists(LIB_PATH), "build the library first"
    L = lib()
    for name in _declared():
        assert hasattr(L, name), name
        assert isinstance(getattr(L, name), ctypes._CFuncPtr)


def test_chunk_plan_host_logic_matches_oracle():
    """tsid_chunk_plan is host-only: no context, no device."""
    from paper_2608_00977_amd import tsid_chunk_plan
    g = np.random.default_rng(2)
    for trial in range(200):
        n = int(g.integers(0, 50))
        counts = g.integers(0, 30, n) * (g.random(n) < 0.7)
        if n and trial % 3 == 0:
            counts[g.integers(0, n)] = 1000
        for K in (1, 2, 7):
            assert np.array_equal(tsid_chunk_plan(counts, n_chunks=K), oracle.chunk_plan(counts, K))
        for cap in (1, 25, 100):
            assert np.array_equal(tsid_chunk_plan(counts, max_entries=cap),
                                  oracle.chunk_plan(counts, max_entries=cap))


def test_create_with_a_device_id_no_runtime_has_is_e_device():
    """tsid_create validates the device id before any device work: an id no
    runtime has (here, and on any box) returns TSID_E_DEVICE and no context."""
    from paper_2608_00977_amd import lib
    L = lib()
    ctx = ctypes.c_void_p()
    st = L.tsid_create(100000, None, 0, ctypes.byref(ctx))
    assert st == 5 and not ctx.value
    assert L.tsid_create(0, None, 0, None) == 1  # out == NULL: TSID_E_INVAL
