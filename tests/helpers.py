"""Test plumbing: hand the same synthetic bytes to the oracle (numpy) and the
HIP library (torch device tensors).  No method arithmetic lives here."""
from __future__ import annotations

import numpy as np
import torch


def np_float(t: torch.Tensor) -> np.ndarray:
    """Exact widening of a bf16/f32 tensor to a float32 numpy array."""
    return t.detach().to("cpu", torch.float32).numpy()


def oracle_state(st: dict) -> dict:
    """numpy copy of a generator/GPU state in the oracle's dictionary form."""
    out = {}
    for key in ("parent", "n_full", "tok_off", "page_off", "n_kept", "page_table", "slot_pos",
                "free_stack"):
        out[key] = st[key].detach().cpu().numpy().astype(np.int64)
    out["free_top"] = np.int64(int(st["free_top"].reshape(-1)[0]))
    out["k"] = np_float(st["k"])
    out["v"] = np_float(st["v"])
    out["page_size"] = int(st["page_size"])
    return out


def oracle_params(p: dict) -> dict:
    return dict(p)
