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


STRUCTS = {"Geom": "arbor_geom_t", "TreeS": "arbor_tree_t", "PoolS": "arbor_pool_t",
           "Params": "arbor_params_t", "Sizes": "arbor_sizes_t",
           "DecodeCredit": "arbor_decode_credit_t", "Timing": "arbor_timing_t",
           "Walk": "arbor_walk_t"}


def test_struct_layouts(tmp_path):
    """Every binding struct has the C compiler's size and field offsets for
    the header's struct (a host C program built with gcc prints them)."""
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "arbor.h"', "int main(void) {"]
    for py, c in STRUCTS.items():
        lines.append(f'  printf("{py} size %zu\\n", sizeof({c}));')
        for name, _ in getattr(L, py)._fields_:
            lines.append(f'  printf("{py} {name} %zu\\n", offsetof({c}, {name}));')
    lines.append("  return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    import subprocess
    subprocess.run(["gcc", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                    "-I", "/opt/rocm/include", str(src), "-o", str(exe)], check=True)
    got = {}
    for line in subprocess.run([str(exe)], check=True, capture_output=True,
                               text=True).stdout.splitlines():
        py, name, val = line.split()
        got[(py, name)] = int(val)
    for py in STRUCTS:
        cls = getattr(L, py)
        assert got[(py, "size")] == ctypes.sizeof(cls), py
        for name, _ in cls._fields_:
            assert got[(py, name)] == getattr(cls, name).offset, (py, name)


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


def test_timing_request_is_validated_on_the_host():
    """A per-call timing request names a known kernel and both events; a bad
    one is refused before anything is enqueued (the geometry is checked
    first, so no tree or pool is needed)."""
    lib = L.load()
    e = ctypes.c_void_p(1)
    for bad in (L.Timing(L.KERNEL_COUNT, e, e),
                L.Timing(-1, e, e), L.Timing(L.KERNEL_SELECT, e, None),
                L.Timing(L.KERNEL_SELECT, None, e)):
        g = L.Geom(32, 8, 4, 128, 16, L.BF16, 1408)
        g.timing = ctypes.pointer(bad)
        assert lib.arbor_select(ctypes.byref(g), None, None, None, None, None, None, None,
                                None) == L.EINVAL


def test_library_keeps_no_timing_state():
    """No entry point other than those of the header is exported: in
    particular no process-wide setter of timing events."""
    lib = L.load()
    assert not hasattr(lib, "arbor_set_kernel_events")


def test_uncertainty_workspace_sizes_on_the_host():
    # the chunked forms need per-chunk partials and, for top-K, K <= 256
    # candidates per chunk: the size grows with the rows and covers them
    small = L.arbor_uncertainty_workspace_size(8, 128256, L.BF16)
    large = L.arbor_uncertainty_workspace_size(85, 128256, L.BF16)
    assert 0 < small < large
    assert large >= 85 * (16 + 4 * 256 + 4)
    assert L.arbor_uncertainty_workspace_size(0, 128256, L.BF16) > 0
    with pytest.raises(ValueError):
        import torch
        L.arbor_uncertainty(torch.zeros(4), 0, None, None, None)


def test_decode_workspace_covers_the_credit_lse():
    # the scored decode keeps a log2 LSE per (leaf, layer, query head) in the
    # shared workspace: more leaves or layers need more bytes
    lib = L.load()
    g = L.Geom(32, 8, 4, 128, 16, L.BF16, 1408)
    a = L.Sizes(85, 22528, 1792, 1, 32, 2, 4, 32)
    b = L.Sizes(85, 22528, 1792, 1, 32, 2, 64, 32)
    na = lib.arbor_workspace_size(ctypes.byref(g), ctypes.byref(a))
    nb = lib.arbor_workspace_size(ctypes.byref(g), ctypes.byref(b))
    assert nb - na >= (64 - 4) * 32 * 32 * 4
