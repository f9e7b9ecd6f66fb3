"""arbor_select_compact (select then compact on the same k in one entry point)
against the oracle's select + compact, and against the two separate entry
points on the same inputs: bit-exact selections, page tables, slot maps,
free stacks and retained K/V bytes.  Nested events on random trees in every
selection mode, blocks over 512 and 1,024 resident tokens (the streamed
selection path), the global sinks, and the error paths, which must leave the
state unchanged."""
import math

import numpy as np
import pytest
import torch

from oracle import arbor_oracle as O
from paper_2605_22106_amd import _lib as L
from paper_2605_22106_amd import synth
from tests.gpu_helpers import assert_same_pool, check_rc, gpu_to_oracle, status, to_gpu, workspace
from tests.helpers import oracle_state

pytestmark = pytest.mark.gpu

PARAMS = dict(alpha_max=math.inf, gamma=2.0, lambda_d=0.1, lambda_delta=0.5, eta=0.8, r_min=0.05,
              k_min=2, l_tail=5, theta=(1.0, 1.0, 1.0), select_mode=0, score_self_window=0)


def _fused(st, kv, A_np, k_np, p):
    N = st["num_tokens"]
    A = torch.tensor(A_np, device="cuda")
    k = torch.tensor(k_np, dtype=torch.int32, device="cuda")
    sel = torch.full((N,), -7, dtype=torch.int32, device="cuda")
    stt = status()
    check_rc(L.arbor_select_compact(kv, A, k, p, sel, stt, workspace(kv)))
    torch.cuda.synchronize()
    return sel.cpu().numpy(), int(stt)


def _separate(st, kv, A_np, k_np, p):
    N = st["num_tokens"]
    A = torch.tensor(A_np, device="cuda")
    k = torch.tensor(k_np, dtype=torch.int32, device="cuda")
    sel = torch.full((N,), -7, dtype=torch.int32, device="cuda")
    stt = status()
    check_rc(L.arbor_select(kv, A, k, p, sel, stt))
    check_rc(L.arbor_compact(kv, k, sel, stt, workspace(kv)))
    torch.cuda.synchronize()
    return sel.cpu().numpy(), int(stt)


def _rand_A(N, seed):
    rng = np.random.default_rng(seed)
    A = (np.round(rng.random(N) * 8) / 8).astype(np.float32)     # ties: lower position wins
    A[rng.random(N) < 0.05] = -0.0
    return A


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("mode,sinks", [(0, 0), (1, 0), (0, 4), (2, 4)])
def test_fused_matches_oracle_and_separate_calls(seed, mode, sinks):
    parent, n_full = synth.random_tree(28, 90, seed, min_tokens=1)
    leaves = [i for i in range(28) if i not in parent]
    st = synth.build_state(parent, n_full, layers=2, kv_heads=2, q_per_kv=2,
                           head_dim=128 if seed % 2 else 64, dtype="bf16" if seed % 2 else "f32",
                           seed=seed, shuffle_pages=True, page_size=16, spare_pages=4,
                           active=leaves[:2])
    kv_f, kv_s = to_gpu(st), to_gpu(st)
    ost = oracle_state(st)
    rng = np.random.default_rng(seed + 70)
    p = dict(PARAMS, select_mode=mode, n_sinks=sinks)
    for event in range(3):                                  # nested events
        A = _rand_A(st["num_tokens"], seed * 10 + event)
        k = np.array([int(rng.integers(0, c + 1)) if rng.random() < 0.7 else c
                      for c in ost["n_kept"]], dtype=np.int32)
        sel_o, so = O.select(ost, A, k, p["l_tail"], mode, n_sinks=sinks)
        assert so == O.OK
        sel_f, sf = _fused(st, kv_f, A, k, p)
        sel_s, ss = _separate(st, kv_s, A, k, p)
        assert sf == L.OK and ss == L.OK
        for i, keep in sel_o.items():
            b = int(ost["tok_off"][i])
            assert sel_f[b:b + len(keep)].tolist() == keep, (event, i)
            assert sel_s[b:b + len(keep)].tolist() == keep, (event, i)
        ost = O.compact(ost, k, sel_o)
        assert_same_pool(gpu_to_oracle(kv_f), ost)
        assert_same_pool(gpu_to_oracle(kv_s), ost)


@pytest.mark.parametrize("mode", [0, 1])
def test_fused_large_blocks(mode):
    # blocks over 512 and 1,024 resident tokens take the streamed selection
    parent = [-1, 0, 0, 0, 0, 0, 2, 6]
    n_full = [64, 600, 1100, 2500, 513, 1025, 40, 33]
    st = synth.build_state(parent, n_full, layers=2, kv_heads=2, q_per_kv=1, head_dim=128,
                           dtype="bf16", seed=19, shuffle_pages=True, spare_pages=8, active=[7])
    kv = to_gpu(st)
    ost = oracle_state(st)
    rng = np.random.default_rng(9 + mode)
    p = dict(PARAMS, select_mode=mode)
    N = st["num_tokens"]
    for event, plan in enumerate([{1: 530, 3: 1800, 4: 513, 5: 1025, 2: 1000},
                                  {1: 100, 3: 700, 4: 12, 5: 1024, 2: 3}]):
        A = (np.round(rng.random(N) * 16) / 16).astype(np.float32)
        k = ost["n_kept"].copy()
        for i, ki in plan.items():
            k[i] = min(ki, int(ost["n_kept"][i]))
        sel_o, so = O.select(ost, A, k, p["l_tail"], mode)
        assert so == O.OK
        sel_g, sg = _fused(st, kv, A, k, p)
        assert sg == L.OK, event
        for i, keep in sel_o.items():
            b = int(ost["tok_off"][i])
            assert sel_g[b:b + len(keep)].tolist() == keep, (event, i)
        ost = O.compact(ost, k, sel_o)
        assert_same_pool(gpu_to_oracle(kv), ost)


def test_fused_errors_leave_the_state_unchanged():
    parent, n_full = synth.random_tree(12, 60, 3, min_tokens=20)
    st = synth.build_state(parent, n_full, layers=2, kv_heads=2, q_per_kv=2, head_dim=64,
                           dtype="f32", seed=3, shuffle_pages=True, page_size=16, spare_pages=4,
                           active=[11])
    kv = to_gpu(st)
    before = gpu_to_oracle(kv)
    N = st["num_tokens"]
    # a NaN in A over a changed block
    A = _rand_A(N, 0)
    A[int(st["tok_off"][2]) + 1] = np.nan
    _, sg = _fused(st, kv, A, np.zeros(12, dtype=np.int32), PARAMS)
    assert sg == L.ENONFINITE
    assert_same_pool(gpu_to_oracle(kv), before)
    # a negative keep-count
    k = np.array(before["n_kept"], dtype=np.int32)
    k[4] = -1
    _, sg = _fused(st, kv, _rand_A(N, 1), k, PARAMS)
    assert sg == L.EINVAL
    assert_same_pool(gpu_to_oracle(kv), before)
