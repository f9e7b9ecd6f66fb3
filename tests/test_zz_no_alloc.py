"""arbor_compact_noalloc (the compaction entry point that allocates nothing and
keeps its scratch in a device array of the library) against arbor_compact
(caller workspace) through the C ABI: identical pools, page tables, slot maps,
resident counts and free stacks, bit for bit, on two calls in a row (the
second on a smaller tree, so the shared scratch holds the larger call's
leftovers), and both against the oracle."""
import ctypes
import math

import numpy as np
import pytest
import torch

from oracle import arbor_oracle as O
from paper_2605_22106_amd import _lib as L
from paper_2605_22106_amd import synth
from tests.gpu_helpers import assert_same_pool, check_rc, gpu_to_oracle, status, to_gpu, workspace
from tests.helpers import oracle_state

PARAMS = dict(alpha_max=math.inf, gamma=2.0, lambda_d=0.1, lambda_delta=0.5, eta=0.8, r_min=0.05,
              k_min=2, l_tail=5, theta=(1.0, 1.0, 1.0), select_mode=0, score_self_window=0)


def _case(seed, V, max_n):
    parent, n_full = synth.random_tree(V, max_n, seed, min_tokens=1)
    st = synth.build_state(parent, n_full, layers=2, kv_heads=2, q_per_kv=1, head_dim=128,
                           dtype="bf16", seed=seed, shuffle_pages=True, spare_pages=4,
                           active=[V - 1])
    rng = np.random.default_rng(seed)
    A = rng.random(st["num_tokens"]).astype(np.float32)
    k = np.array([int(rng.integers(0, n + 1)) if rng.random() < 0.7 else n for n in n_full],
                 dtype=np.int32)
    return st, A, k


@pytest.mark.gpu
def test_noalloc_compaction_matches_the_workspace_entry_point():
    # the larger tree first, then a smaller one
    for seed, V, max_n in ((21, 60, 700), (22, 9, 40)):
        st, A_np, k_np = _case(seed, V, max_n)
        kv_ws, kv_na = to_gpu(st), to_gpu(st)
        N = st["num_tokens"]
        A = torch.tensor(A_np, device="cuda")
        k = torch.tensor(k_np, device="cuda")
        sel = torch.full((N,), -7, dtype=torch.int32, device="cuda")
        s_ws, s_na = status(), status()
        check_rc(L.arbor_select(kv_ws, A, k, PARAMS, sel, s_ws))
        check_rc(L.arbor_compact(kv_ws, k, sel, s_ws, workspace(kv_ws)))
        check_rc(L.arbor_compact_noalloc(kv_na, k, sel, s_na))
        torch.cuda.synchronize()
        assert int(s_ws) == int(s_na) == L.OK, seed
        got, ref = gpu_to_oracle(kv_na), gpu_to_oracle(kv_ws)
        assert_same_pool(got, ref)
        ost = oracle_state(st)
        sel_o, _ = O.select(ost, A_np, k_np, PARAMS["l_tail"])
        assert_same_pool(got, O.compact(ost, k_np, sel_o))


def test_noalloc_refuses_trees_beyond_its_scratch_on_the_host():
    """A tree whose scratch would exceed the fixed array is refused before any
    device work (no GPU needed: the check precedes every HIP call)."""
    lib = L.load()
    g = L.Geom(1, 1, 1, 64, 16, L.F32, 1)
    fake = ctypes.c_void_p(256)
    t = L.TreeS(1, 3_000_000, fake, fake, fake, fake, fake, fake)
    p = L.PoolS(fake, fake, fake, fake, fake)
    rc = lib.arbor_compact_noalloc(ctypes.byref(g), ctypes.byref(t), ctypes.byref(p), fake, fake,
                                   fake, None)
    assert rc == L.EWORKSPACE
