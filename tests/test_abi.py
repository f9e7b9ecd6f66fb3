"""The C-ABI library loads and exports every entry point of include/arbor.h
(host-only checks; no kernel is launched)."""
import ctypes
import os
import re

import pytest

from paper_2605_22106_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "arbor.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(arbor_[a-z_]+)\s*\(", src)))


def test_header_matches_binding():
    assert declared_functions() == sorted(L.exported_symbols())


def test_library_exports_every_symbol():
    lib = L.load()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_struct_layouts():
    assert ctypes.sizeof(L.Geom) == 32
    assert ctypes.sizeof(L.TreeS) == 64
    assert ctypes.sizeof(L.PoolS) == 40
    assert ctypes.sizeof(L.Params) == 88
    assert ctypes.sizeof(L.Sizes) == 48


def test_strerror_and_workspace_size_are_host_only():
    assert L.arbor_strerror(L.ENOPAGES) == "not enough free pages"
    assert L.arbor_strerror(12345) == "unknown status"
    lib = L.load()
    g = L.Geom(32, 8, 4, 128, 16, L.BF16, 1408)
    sz = L.Sizes(85, 22528, 1792, 85, 32, 2, 4, 32)
    n = lib.arbor_workspace_size(ctypes.byref(g), ctypes.byref(sz))
    assert n > 22528 * 16


def test_product_path_refuses_cpu_tensors():
    import torch
    with pytest.raises(ValueError):
        L._dev(torch.zeros(3), "x")


def test_kernel_events_setter_validates_on_the_host():
    lib = L.load()
    assert lib.arbor_set_kernel_events(L.KERNEL_SCORE_ATTN, None, None) == L.OK
    assert lib.arbor_set_kernel_events(4, None, None) == L.EINVAL
    assert lib.arbor_set_kernel_events(-1, None, None) == L.EINVAL
    # one of the two events missing
    assert lib.arbor_set_kernel_events(L.KERNEL_DECODE_ATTN, ctypes.c_void_p(1), None) == L.EINVAL
