"""GPU parity of kernel branches that only large or unusual inputs reach.

* selection and compaction of blocks with more than 512 and more than 1,024
  resident tokens (the streamed selection, the compaction plan's source
  search in global memory), in both selection modes, over nested events;
* allocation with gamma = 1 and gamma = 3, with -0 scores under Pressure, and
  with scores outside [0, 1];
* scoring and decode attention on the 9,841-node deep tree (branching 3,
  depth 8, 64 tokens per node), beyond the node counts that the score setup
  (2,048) and the decode plan (4,096) keep in LDS.  The tree and token counts
  are those of the deep configuration; the pool has 2 layers and 2 KV heads
  (G = 4) so that the oracle can replay the sampled observers in test time.

Bars as in the other parity tests: bit-exact for counts, selections, page
tables, slot maps, free stacks and K/V bytes; 1e-4 relative for A, a, s;
2e-3 absolute for fp32 decode outputs.
"""
import math

import numpy as np
import pytest
import torch

from oracle import arbor_oracle as O
from paper_2605_22106_amd import _lib as L
from paper_2605_22106_amd import synth
from tests.gpu_helpers import assert_same_pool, check_rc, gpu_to_oracle, status, to_gpu, workspace
from tests.helpers import np_float, oracle_state

pytestmark = pytest.mark.gpu

PARAMS = dict(alpha_max=math.inf, gamma=2.0, lambda_d=0.1, lambda_delta=0.5, eta=0.8, r_min=0.05,
              k_min=2, l_tail=5, theta=(1.0, 1.0, 1.0), select_mode=0, score_self_window=0)


def _close(g, o, rel=1e-4, atol=1e-30):
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    bad = np.abs(g - o) > rel * np.abs(o) + atol
    assert not bad.any(), (np.nonzero(bad)[0][:10], g[bad][:5], o[bad][:5])


# --------------------------------------------------------------------------- large blocks
@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("f32", 64)])
def test_select_compact_large_blocks(mode, dtype, d):
    # root, four large off-path blocks (513 .. 2,500 tokens) and the active chain
    parent = [-1, 0, 0, 0, 0, 0, 2, 6]
    n_full = [64, 600, 1100, 2500, 513, 1025, 40, 33]
    st = synth.build_state(parent, n_full, layers=2, kv_heads=2, q_per_kv=1, head_dim=d,
                           dtype=dtype, seed=17, shuffle_pages=True, spare_pages=8, active=[7])
    kv = to_gpu(st)
    ost = oracle_state(st)
    rng = np.random.default_rng(5 + mode)
    p = dict(PARAMS, select_mode=mode)
    N = st["num_tokens"]
    # first event keeps the large blocks above 512 / 1,024 resident tokens, the
    # second goes below
    plans = [{1: 530, 3: 1800, 4: 513, 5: 1025, 2: 1000},
             {1: 100, 3: 700, 4: 12, 5: 1024, 2: 3}]
    for event, plan in enumerate(plans):
        A = rng.random(N).astype(np.float32)
        A = (np.round(A * 16) / 16).astype(np.float32)       # many ties: lower position wins
        A[rng.random(N) < 0.05] = -0.0
        k = ost["n_kept"].copy()
        for i, ki in plan.items():
            k[i] = min(ki, int(ost["n_kept"][i]))
        sel_o, so = O.select(ost, A, k, p["l_tail"], mode)
        assert so == O.OK
        At = torch.tensor(A, device="cuda")
        kt = torch.tensor(k, dtype=torch.int32, device="cuda")
        sel = torch.full((N,), -7, dtype=torch.int32, device="cuda")
        stt = status()
        check_rc(L.arbor_select(kv, At, kt, p, sel, stt))
        check_rc(L.arbor_compact(kv, kt, sel, stt, workspace(kv)))
        torch.cuda.synchronize()
        assert int(stt) == L.OK, event
        sel_g = sel.cpu().numpy()
        for i, keep in sel_o.items():
            b = int(ost["tok_off"][i])
            assert sel_g[b:b + len(keep)].tolist() == keep, (event, i)
        ost = O.compact(ost, k, sel_o)
        assert_same_pool(gpu_to_oracle(kv), ost)


# --------------------------------------------------------------------------- allocate
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


@pytest.mark.parametrize("gamma", [1.0, 3.0])
@pytest.mark.parametrize("seed", range(4))
def test_allocate_gamma_and_negative_zero(gamma, seed):
    """Eq. 2 with gamma = 1 and 3, ties between blocks, -0 scores; budgets from
    deep Pressure to none."""
    V = 60
    parent, n_full = synth.random_tree(V, 50, seed + 40, min_tokens=1)
    leaves = [i for i in range(V) if i not in parent]
    rng = np.random.default_rng(seed)
    active = sorted(rng.choice(leaves, size=3, replace=False).tolist())
    st = synth.build_state(parent, n_full, layers=1, kv_heads=1, q_per_kv=1, head_dim=64,
                           dtype="f32", seed=seed, active=active)
    kv = to_gpu(st)
    n_full = st["n_full"].numpy()
    n_kept = np.array([int(rng.integers(0, n + 1)) if rng.random() < 0.3 else n for n in n_full])
    kv.n_kept.copy_(torch.tensor(n_kept, dtype=torch.int32))
    s = rng.random(V).astype(np.float32)
    s[rng.random(V) < 0.15] = np.float32(-0.0)
    s[rng.random(V) < 0.1] = 0.0
    s[:6] = s[6]                                  # exact weight ties
    p = dict(PARAMS, gamma=gamma)
    pressure = 0
    for rho in (0.05, 0.1, 0.2, 0.35, 0.6, 1.0):
        budget = int(rho * n_full.sum())
        k_o, d_o, on_o, st_o = O.allocate(parent, n_full, n_kept, active, budget, s, p)
        k, dl, onp, sg = _alloc_gpu(kv, active, budget, s, p)
        assert sg == st_o, rho
        assert np.array_equal(k, k_o), rho
        assert np.array_equal(dl, d_o)
        assert np.array_equal(onp, on_o)
        off = [i for i in range(V) if not on_o[i]]
        path = sum(int(n_full[i]) for i in range(V) if on_o[i])
        pressure += sum(O.floor_count(n_full[i], n_kept[i], p) for i in off) > budget - path
    assert pressure > 0, "some budgets reach the Pressure branch"


def test_allocate_scores_outside_the_unit_interval():
    parent, n_full = synth.complete_tree(2, 2, 20, 10)
    st = synth.build_state(parent, n_full, layers=1, kv_heads=1, q_per_kv=1, head_dim=64,
                           dtype="f32", seed=0, active=[3])
    kv = to_gpu(st)
    base = np.full(7, 0.5, np.float32)
    for node, bad in ((2, 1.5), (2, -0.25), (2, np.nan), (1, 7.0)):
        s = base.copy()
        s[node] = bad
        _, _, _, so = O.allocate(parent, n_full, n_full, [3], 40, s, PARAMS)
        k, _, _, sg = _alloc_gpu(kv, [3], 40, s, PARAMS)
        assert sg == so, (node, bad)


# --------------------------------------------------------------------------- deep tree
@pytest.fixture(scope="module")
def deep_tree():
    cfg = synth.CONFIGS["deep"]
    V = sum(3 ** l for l in range(9))
    rng = np.random.default_rng(31)
    # sampled observers: the root, inner nodes of every depth, and leaves in
    # sibling groups (which share their whole ancestor chain)
    depth_start = [sum(3 ** l for l in range(k)) for k in range(10)]
    obs = [0]
    for dd in range(1, 8):
        obs += sorted(rng.choice(np.arange(depth_start[dd], depth_start[dd + 1]), 3,
                                 replace=False).tolist())
    first = depth_start[8]
    for g in rng.choice(np.arange(first, V, 3), 6, replace=False):
        obs += [int(g), int(g) + 1, int(g) + 2]
    obs = sorted(set(obs))
    st = synth.build_config(cfg, device="cuda", layers=2, kv_heads=2, slice_layers=[0, 1],
                            observers=obs, host_store=False, decode_queries=False)
    leaves = sorted(rng.choice(np.arange(first, V), 12, replace=False).tolist())
    kv = L.kv_state_from(st, "cuda")
    return st, kv, obs, leaves


@pytest.mark.parametrize("V", [700, 2600])
def test_score_more_observers_than_one_prep_launch(V):
    """More than 512 observers: the setup and the sub-page tables run as two
    launches (the setup walking the tree from LDS up to 2,048 nodes, from
    global memory beyond)."""
    parent, n_full = synth.random_tree(V, 12, 40 + V, min_tokens=1)
    rng = np.random.default_rng(V)
    obs = sorted(rng.choice(V, 600, replace=False).tolist())
    st = synth.build_state(parent, n_full, layers=1, kv_heads=1, q_per_kv=1, head_dim=64,
                           dtype="bf16", seed=V, shuffle_pages=True, page_size=16, window=4,
                           observers=obs, active=[obs[-1]], host_store=False,
                           decode_queries=False)
    kv = to_gpu(st)
    ost = oracle_state(st)
    p = dict(PARAMS, theta=(0.5, -1.0, 2.0))
    N = st["num_tokens"]
    ws = workspace(kv, max_observers=len(obs), window=4, n_slice=len(st["slice_layers"]))
    A = torch.zeros(N, device="cuda")
    rows = torch.zeros(V, dtype=torch.int64, device="cuda")
    a = torch.empty(V, device="cuda")
    s = torch.empty(V, device="cuda")
    stt = status()
    check_rc(L.arbor_score(kv, st["observers"].cuda(), st["q_win"].cuda().contiguous(), 4,
                           st["slice_layers"], st["v_sig"].cuda(), st["u_sig"].cuda(), A, rows,
                           a, s, p, stt, ws))
    torch.cuda.synchronize()
    assert int(stt) == L.OK
    Ao, ro, ao, so = O.score(ost, obs, np_float(st["q_win"]), 4, st["slice_layers"], 1,
                             st["v_sig"].numpy(), st["u_sig"].numpy(), np.zeros(N, np.float32),
                             np.zeros(V, np.int64), theta=p["theta"])
    _close(A.cpu().numpy(), Ao)
    assert np.array_equal(rows.cpu().numpy(), ro)
    _close(a.cpu().numpy(), ao)
    _close(s.cpu().numpy(), so)


def test_deep_tree_score_sampled_observers(deep_tree):
    st, kv, obs, _ = deep_tree
    V, N = kv.num_nodes, kv.num_tokens
    assert V == 9841 and N == 630784
    p = dict(st["params"])
    ws = workspace(kv, max_context=1024 + 8 * 64, max_observers=len(obs), window=st["window"],
                   n_slice=2)
    A = torch.zeros(N, device="cuda")
    rows = torch.zeros(V, dtype=torch.int64, device="cuda")
    a = torch.empty(V, device="cuda")
    s = torch.empty(V, device="cuda")
    stt = status()
    check_rc(L.arbor_score(kv, st["observers"].cuda(), st["q_win"].cuda().contiguous(),
                           st["window"], [0, 1], st["v_sig"].cuda(), st["u_sig"].cuda(), A, rows,
                           a, s, p, stt, ws))
    torch.cuda.synchronize()
    assert int(stt) == L.OK
    ost = oracle_state({**st, "k": kv.k, "v": kv.v[:, :1, :, :, :1]})
    Ao, ro, ao, so = O.score(ost, obs, np_float(st["q_win"]), st["window"], [0, 1],
                             kv.q_per_kv, st["v_sig"].numpy(), st["u_sig"].numpy(),
                             np.zeros(N, np.float32), np.zeros(V, np.int64), theta=p["theta"])
    _close(A.cpu().numpy(), Ao)
    assert np.array_equal(rows.cpu().numpy(), ro)
    _close(a.cpu().numpy(), ao)
    _close(s.cpu().numpy(), so)


def test_deep_tree_decode_after_eviction(deep_tree):
    st, kv, _, leaves = deep_tree
    V, N = kv.num_nodes, kv.num_tokens
    # an eviction event first (random A and k), so chains are ragged
    rng = np.random.default_rng(8)
    ost = oracle_state({**st, "k": kv.k, "v": kv.v})
    A = rng.random(N).astype(np.float32)
    k = ost["n_kept"].copy()
    lower = rng.random(V) < 0.5
    k[lower] = rng.integers(0, k[lower] + 1)
    sel_o, _ = O.select(ost, A, k, 8)
    sel = torch.full((N,), -7, dtype=torch.int32, device="cuda")
    stt = status()
    kt = torch.tensor(k, dtype=torch.int32, device="cuda")
    check_rc(L.arbor_select(kv, torch.tensor(A, device="cuda"), kt, st["params"], sel, stt))
    check_rc(L.arbor_compact(kv, kt, sel, stt, workspace(kv)))
    torch.cuda.synchronize()
    assert int(stt) == L.OK
    ost = O.compact(ost, k, sel_o)
    Hq = kv.kv_heads * kv.q_per_kv
    g = torch.Generator(device="cuda").manual_seed(3)
    q = torch.randn((len(leaves), 2, Hq, kv.head_dim), generator=g, device="cuda").to(torch.bfloat16)
    out = torch.empty((len(leaves), 2, Hq, kv.head_dim), device="cuda")
    lse = torch.empty((len(leaves), 2, Hq), device="cuda")
    lt = torch.tensor(leaves, dtype=torch.int32, device="cuda")
    check_rc(L.arbor_tree_decode_attn(kv, lt, 0, 2, q, out, lse, 0.0, stt,
                                      workspace(kv, max_leaves=len(leaves), max_layers=2)))
    torch.cuda.synchronize()
    assert int(stt) == L.OK
    now = gpu_to_oracle(kv)
    for key in ("n_kept", "page_table", "slot_pos"):
        assert np.array_equal(now[key], ost[key]), key
    o_o, lse_o = O.tree_decode_attn(now, leaves, 0, 2, np_float(q), kv.q_per_kv)
    assert np.max(np.abs(out.cpu().numpy() - o_o)) <= 2e-3
    fin = np.isfinite(lse_o)
    assert np.max(np.abs(lse.cpu().numpy()[fin] - lse_o[fin])) <= 1e-4 * np.abs(lse_o[fin]).max()
