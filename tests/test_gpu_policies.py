"""GPU parity of the policy variants against the oracle:

* floor protection of Path* blocks (invariant (i) with a floor k_protect):
  keep-counts bit-exact over budgets from deep Pressure to none, with and
  without rehydration;
* the global sinks of the root prompt and the three intra-block rules of
  Table 7 (sinks + tail + heavy hitters, tail only, sinks + tail), with the
  root cut, over nested events, for a root held in registers (<= 512 resident
  tokens) and a root streamed from memory (> 512);
* one whole floor-protection event: allocate -> rehydrate -> select ->
  compact, state bit-exact against the oracle's sequence.
"""
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


def _alloc_gpu(kv, active, budget, s, p):
    V = kv.num_nodes
    k = torch.empty(V, dtype=torch.int32, device="cuda")
    dl = torch.empty_like(k)
    onp = torch.empty(V, dtype=torch.uint8, device="cuda")
    stt = status()
    check_rc(L.arbor_allocate(kv, torch.tensor(active, dtype=torch.int32, device="cuda"), budget,
                              torch.tensor(s, device="cuda"), p, k, dl, onp, stt, workspace(kv)))
    torch.cuda.synchronize()
    return k.cpu().numpy(), dl.cpu().numpy(), onp.cpu().numpy(), int(stt)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("rehydrate", [1, 0])
def test_allocate_floor_protection(seed, rehydrate):
    V = 60 if seed < 4 else 700                     # per-node state in LDS, then in memory
    parent, n_full = synth.random_tree(V, 50, seed + 90, min_tokens=1)
    leaves = [i for i in range(V) if i not in set(parent)]
    rng = np.random.default_rng(seed)
    active = sorted(rng.choice(leaves, size=3, replace=False).tolist())
    st = synth.build_state(parent, n_full, layers=1, kv_heads=1, q_per_kv=1, head_dim=64,
                           dtype="f32", seed=seed, active=active)
    kv = to_gpu(st)
    n_full = st["n_full"].numpy()
    n_kept = np.array([int(rng.integers(0, n + 1)) if rng.random() < 0.4 else n for n in n_full])
    kv.n_kept.copy_(torch.tensor(n_kept, dtype=torch.int32))
    s = rng.random(V).astype(np.float32)
    s[:6] = s[6]                                    # exact weight ties
    s[rng.random(V) < 0.1] = 0.0
    p = dict(PARAMS, k_protect=[4, 12, 30][seed % 3], lazy_rehydration=rehydrate)
    if seed % 2:
        p["alpha_max"] = 0.6
    seen = set()
    for rho in (0.05, 0.15, 0.3, 0.5, 0.8, 1.0):
        budget = int(rho * n_full.sum())
        k_o, d_o, on_o, st_o = O.allocate(parent, n_full, n_kept, active, budget, s, p)
        k, dl, onp, sg = _alloc_gpu(kv, active, budget, s, p)
        assert sg == st_o, rho
        assert np.array_equal(k, k_o), rho
        assert np.array_equal(dl, d_o)
        assert np.array_equal(onp, on_o)
        seen.add(st_o)
    assert O.OK in seen


def _select_compact(kv, A_np, k_np, p):
    N = kv.num_tokens
    A = torch.tensor(A_np, device="cuda")
    k = torch.tensor(k_np, dtype=torch.int32, device="cuda")
    sel = torch.full((N,), -7, dtype=torch.int32, device="cuda")
    stt = status()
    check_rc(L.arbor_select(kv, A, k, p, sel, stt))
    check_rc(L.arbor_compact(kv, k, sel, stt, workspace(kv)))
    torch.cuda.synchronize()
    return sel.cpu().numpy(), int(stt)


@pytest.mark.parametrize("mode", [0, 1, 2])
@pytest.mark.parametrize("root", [300, 1400])
def test_select_sinks_and_rules(mode, root):
    parent = [-1, 0, 0, 1, 1, 2]
    n_full = [root, 70, 90, 40, 33, 61]
    st = synth.build_state(parent, n_full, layers=2, kv_heads=2, q_per_kv=1, head_dim=128,
                           dtype="bf16", seed=mode + root, shuffle_pages=True, spare_pages=4,
                           active=[3])
    kv = to_gpu(st)
    ost = oracle_state(st)
    rng = np.random.default_rng(mode * 7 + root)
    p = dict(PARAMS, select_mode=mode)
    N = st["num_tokens"]
    # root cut to: fewer than its sinks, sinks + part of the tail, deep heavy
    # selections; the sink count varies between events
    for event, (k0, n_sinks) in enumerate(((root * 3 // 4, 24), (root // 3, 64), (40, 8),
                                           (5, 16))):
        A = (np.round(rng.random(N) * 12) / 12).astype(np.float32)
        A[rng.random(N) < 0.05] = -0.0
        k = np.array([min(int(c), int(rng.integers(0, int(c) + 1))) for c in ost["n_kept"]])
        k[0] = min(k0, int(ost["n_kept"][0]))
        p["n_sinks"] = n_sinks
        sel_o, so = O.select(ost, A, k, p["l_tail"], mode, n_sinks=n_sinks)
        assert so == O.OK
        sel_g, sg = _select_compact(kv, A, k, p)
        assert sg == L.OK, event
        for i, keep in sel_o.items():
            b = int(ost["tok_off"][i])
            assert sel_g[b:b + len(keep)].tolist() == keep, (event, i)
        ost = O.compact(ost, k, sel_o)
        assert_same_pool(gpu_to_oracle(kv), ost)


@pytest.mark.parametrize("seed", range(3))
def test_floor_protection_event(seed):
    """allocate (floor protection, sinks) -> rehydrate -> select -> compact
    after a first event and a move of the active leaf, bit-exact against the
    oracle's sequence: Path* blocks are restored, then cut to their keep-count
    with the root's sinks kept."""
    V = 30
    parent, n_full = synth.random_tree(V, 90, seed + 120, min_tokens=8)
    n_full[0] = 200
    leaves = [i for i in range(V) if i not in set(parent)]
    rng = np.random.default_rng(seed)
    a0, a1 = rng.choice(leaves, size=2, replace=False).tolist()
    st = synth.build_state(parent, n_full, layers=2, kv_heads=2, q_per_kv=1, head_dim=128,
                           dtype="bf16", seed=seed, shuffle_pages=True, spare_pages=16,
                           active=[a0])
    kv = to_gpu(st)
    ost = oracle_state(st)
    hk = st["host_k"].pin_memory()
    hv = st["host_v"].pin_memory()
    hk_o, hv_o = hk.float().numpy(), hv.float().numpy()
    p = dict(PARAMS, k_protect=24, n_sinks=6)
    s = rng.random(V).astype(np.float32)
    N = st["num_tokens"]
    ws = workspace(kv)
    for event, leaf in enumerate((a0, a1)):
        budget = int(0.3 * N)
        A = rng.random(N).astype(np.float32)
        k_o, _, on_o, st_o = O.allocate(ost["parent"], ost["n_full"], ost["n_kept"], [leaf],
                                        budget, s, p)
        k = torch.empty(V, dtype=torch.int32, device="cuda")
        onp = torch.empty(V, dtype=torch.uint8, device="cuda")
        stt = status()
        check_rc(L.arbor_allocate(kv, torch.tensor([leaf], dtype=torch.int32, device="cuda"),
                                  budget, torch.tensor(s, device="cuda"), p, k,
                                  torch.empty_like(k), onp, stt, ws))
        check_rc(L.arbor_rehydrate(kv, onp, hk, hv, stt, ws))
        sel = torch.full((N,), -7, dtype=torch.int32, device="cuda")
        check_rc(L.arbor_select(kv, torch.tensor(A, device="cuda"), k, p, sel, stt))
        check_rc(L.arbor_compact(kv, k, sel, stt, ws))
        torch.cuda.synchronize()
        assert int(stt) == st_o, event
        assert np.array_equal(k.cpu().numpy(), k_o), event
        ost, rs = O.rehydrate(ost, on_o, hk_o, hv_o)
        assert rs == O.OK
        sel_o, so = O.select(ost, A, k_o, p["l_tail"], p["select_mode"], n_sinks=p["n_sinks"])
        assert so == O.OK
        ost = O.compact(ost, k_o, sel_o)
        assert_same_pool(gpu_to_oracle(kv), ost)
        # Path* blocks sit at their floor or above; the root keeps its sinks
        for i in np.nonzero(on_o)[0]:
            assert int(ost["n_kept"][i]) >= min(int(ost["n_full"][i]), p["k_protect"])
        root = [r[3] for r in O.retained(ost, 0)]
        assert root[:p["n_sinks"]] == list(range(p["n_sinks"]))
