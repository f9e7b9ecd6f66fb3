"""Plumbing for the GPU parity tests: run the HIP library on the same bytes the
oracle sees and bring its state back as numpy."""
from __future__ import annotations

import numpy as np
import torch

from paper_2605_22106_amd import _lib as L
from tests.helpers import oracle_state


def to_gpu(st: dict) -> L.KVState:
    return L.kv_state_from(st, "cuda")


def gpu_to_oracle(kv: L.KVState) -> dict:
    d = dict(parent=kv.parent, n_full=kv.n_full, tok_off=kv.tok_off, page_off=kv.page_off,
             n_kept=kv.n_kept, page_table=kv.page_table, slot_pos=kv.slot_pos,
             free_stack=kv.free_stack, free_top=kv.free_top, k=kv.k, v=kv.v,
             page_size=kv.page_size)
    return oracle_state(d)


def workspace(kv: L.KVState, **kw) -> torch.Tensor:
    n = L.arbor_workspace_size(kv, **kw)
    return torch.empty(n, dtype=torch.uint8, device="cuda")


def status() -> torch.Tensor:
    return torch.zeros(1, dtype=torch.int32, device="cuda")


def check_rc(rc: int):
    assert rc == L.OK, f"host-side error {rc}: {L.arbor_strerror(rc)}"


def assert_same_pool(a: dict, b: dict, sel_nodes=None):
    """Bitwise equality of two pool states on every resident slot."""
    for key in ("n_kept", "page_table", "slot_pos"):
        assert np.array_equal(a[key], b[key]), key
    assert int(a["free_top"]) == int(b["free_top"])
    top = int(a["free_top"])
    assert np.array_equal(a["free_stack"][:top], b["free_stack"][:top])
    P = a["page_size"]
    used = set()
    for i in range(len(a["n_kept"])):
        po = int(a["page_off"][i])
        for s in range(int(a["n_kept"][i])):
            used.add((int(a["page_table"][po + s // P]), s % P))
    pages = np.array(sorted({p for p, _ in used}))
    if len(pages):
        mask = np.zeros((a["k"].shape[1], P), dtype=bool)
        for p_, r_ in used:
            mask[p_, r_] = True
        ka = a["k"].transpose(1, 3, 0, 2, 4)[mask]
        kb = b["k"].transpose(1, 3, 0, 2, 4)[mask]
        va = a["v"].transpose(1, 3, 0, 2, 4)[mask]
        vb = b["v"].transpose(1, 3, 0, 2, 4)[mask]
        assert np.array_equal(ka.view(np.uint32), kb.view(np.uint32))
        assert np.array_equal(va.view(np.uint32), vb.view(np.uint32))
