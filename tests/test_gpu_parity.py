"""GPU parity of every step of the path against the CPU oracle, stage by stage
on shared inputs (the same A, k, s and pool bytes are handed to both sides).

Bars: bit-exact for keep-counts, distances, Path*, selections, page tables,
slot maps, free stacks and retained K/V bytes; |g - o| <= 1e-4 |o| + 1e-30 for
A, a, s (fp32); |g - o| <= 2e-3 for fp32 decode outputs, and for bf16 outputs
the larger of 2e-3 and one bf16 ulp of the oracle value rounded to bf16.
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


def rand_tree_state(seed, V=24, max_n=70, min_n=1, L_=2, Hkv=2, G=2, d=128, dtype="bf16",
                    window=8, active=None, spare=4, heavy=0.05):
    parent, n_full = synth.random_tree(V, max_n, seed, min_tokens=min_n)
    if active is None:
        leaves = [i for i in range(V) if i not in parent]
        rng = np.random.default_rng(seed)
        active = sorted(rng.choice(leaves, size=min(3, len(leaves)), replace=False).tolist())
    return synth.build_state(parent, n_full, layers=L_, kv_heads=Hkv, q_per_kv=G, head_dim=d,
                             dtype=dtype, seed=seed, shuffle_pages=True, page_size=16,
                             spare_pages=spare, window=window, active=active, heavy_frac=heavy)


def rand_A(N, seed, ties=True):
    rng = np.random.default_rng(seed)
    A = rng.random(N).astype(np.float32)
    if ties:
        A = (np.round(A * 8) / 8).astype(np.float32)
        A[rng.random(N) < 0.05] = -0.0
    return A


# --------------------------------------------------------------------------- allocate
@pytest.mark.parametrize("seed", range(10))
def test_allocate_bit_exact(seed):
    run_allocate_bit_exact(seed, dict(PARAMS))


@pytest.mark.parametrize("seed", range(4))
def test_allocate_bit_exact_without_rehydration(seed):
    run_allocate_bit_exact(seed + 50, dict(PARAMS, lazy_rehydration=0))


def run_allocate_bit_exact(seed, base):
    st = rand_tree_state(seed, V=60, max_n=50)
    kv = to_gpu(st)
    rng = np.random.default_rng(seed)
    V = kv.num_nodes
    n_full = st["n_full"].numpy()
    n_kept = np.array([int(rng.integers(0, n + 1)) if rng.random() < 0.3 else n for n in n_full])
    kv.n_kept.copy_(torch.tensor(n_kept, dtype=torch.int32))
    s = rng.random(V).astype(np.float32)
    s[rng.random(V) < 0.1] = 0.0
    s[:5] = s[5]                                  # exact weight ties
    p = dict(base)
    if seed % 3 == 1:
        p["alpha_max"] = 0.9
    ws = workspace(kv)
    active = st["active"].cuda()
    for rho in (0.1, 0.3, 0.5, 0.8, 1.0):
        budget = int(rho * st["num_tokens"])
        k_o, d_o, on_o, st_o = O.allocate(st["parent"].numpy(), n_full, n_kept,
                                          st["active"].numpy(), budget, s, p)
        k = torch.empty(V, dtype=torch.int32, device="cuda")
        dl = torch.empty_like(k)
        onp = torch.empty(V, dtype=torch.uint8, device="cuda")
        stt = status()
        check_rc(L.arbor_allocate(kv, active, budget, torch.tensor(s, device="cuda"), p, k, dl,
                                  onp, stt, ws))
        torch.cuda.synchronize()
        assert int(stt) == st_o, rho
        assert np.array_equal(k.cpu().numpy(), k_o), rho
        assert np.array_equal(dl.cpu().numpy(), d_o)
        assert np.array_equal(onp.cpu().numpy(), on_o)


@pytest.mark.parametrize("V,max_n,seed", [(300, 400, 0), (300, 400, 1), (1500, 100, 2),
                                           (10240, 20, 4), (12000, 40, 3)])
def test_allocate_large_bracketed(V, max_n, seed):
    """Tens of thousands of prices, so the order statistic is bracketed by the
    rounded counts before the prices in the bracket are listed.  Node sizes come
    from a small set and weights are rounded to 1/8, so whole runs of prices tie
    exactly; alpha_max both open and binding.  V = 300 keeps the per-node state
    in LDS; V = 1500 and V = 10240 (the largest such tree) keep only the tree's
    geometry there; V = 12000 keeps everything in the workspace."""
    parent, _ = synth.random_tree(V, max_n, seed)
    rng = np.random.default_rng(seed)
    sizes = np.array([max_n // 4, max_n // 2, max_n])
    n_full = [int(x) for x in rng.choice(sizes, size=V)]
    leaves = [i for i in range(V) if i not in set(parent)]
    active = sorted(rng.choice(leaves, size=4, replace=False).tolist())
    st = synth.build_state(parent, n_full, layers=1, kv_heads=1, q_per_kv=1, head_dim=64,
                           dtype="f32", seed=seed, active=active)
    kv = to_gpu(st)
    n_full = st["n_full"].numpy()
    n_kept = np.array([int(rng.integers(n // 2, n + 1)) if rng.random() < 0.3 else n
                       for n in n_full])
    kv.n_kept.copy_(torch.tensor(n_kept, dtype=torch.int32))
    s = (np.round(rng.random(V) * 8) / 8).astype(np.float32)
    ws = workspace(kv)
    act = torch.tensor(active, dtype=torch.int32, device="cuda")
    total = int(n_kept.sum())
    for amax in (math.inf, 0.5):
        p = dict(PARAMS, alpha_max=amax)
        for rho in (0.05, 0.2, 0.5, 0.9):
            budget = int(rho * total)
            k_o, d_o, on_o, st_o = O.allocate(st["parent"].numpy(), n_full, n_kept, active,
                                              budget, s, p)
            k = torch.empty(V, dtype=torch.int32, device="cuda")
            dl = torch.empty_like(k)
            onp = torch.empty(V, dtype=torch.uint8, device="cuda")
            stt = status()
            check_rc(L.arbor_allocate(kv, act, budget, torch.tensor(s, device="cuda"), p, k, dl,
                                      onp, stt, ws))
            torch.cuda.synchronize()
            assert int(stt) == st_o, (amax, rho)
            assert np.array_equal(k.cpu().numpy(), k_o), (amax, rho)
            assert np.array_equal(dl.cpu().numpy(), d_o)
            assert np.array_equal(onp.cpu().numpy(), on_o)


def test_allocate_tiny_config_over_budget():
    st = synth.build_config("tiny")
    kv = to_gpu(st)
    s = torch.full((7,), 0.5, device="cuda")
    k = torch.empty(7, dtype=torch.int32, device="cuda")
    dl = torch.empty_like(k)
    onp = torch.empty(7, dtype=torch.uint8, device="cuda")
    stt = status()
    check_rc(L.arbor_allocate(kv, st["active"].cuda(), st["budget"], s, st["params"], k, dl, onp,
                              stt, workspace(kv)))
    torch.cuda.synchronize()
    assert int(stt) == L.OVER_BUDGET
    assert k.cpu().tolist() == [64, 32, 2, 32, 2, 2, 2]


def test_allocate_rejects_malformed_tree():
    st = rand_tree_state(1, V=10)
    kv = to_gpu(st)
    bad = kv.parent.clone()
    bad[5] = 7                                         # parent not below the child
    kv.parent = bad
    k = torch.empty(10, dtype=torch.int32, device="cuda")
    stt = status()
    check_rc(L.arbor_allocate(kv, st["active"].cuda(), 100, torch.rand(10, device="cuda"), PARAMS,
                              k, torch.empty_like(k), torch.empty(10, dtype=torch.uint8,
                                                                  device="cuda"), stt,
                              workspace(kv)))
    torch.cuda.synchronize()
    assert int(stt) == L.EINVAL


# --------------------------------------------------------------------------- select + compact
def _event(st, kv, A_np, k_np, p):
    """select + compact on the GPU; returns (sel_pos, status)."""
    N = st["num_tokens"]
    A = torch.tensor(A_np, device="cuda")
    k = torch.tensor(k_np, dtype=torch.int32, device="cuda")
    sel = torch.full((N,), -7, dtype=torch.int32, device="cuda")
    stt = status()
    check_rc(L.arbor_select(kv, A, k, p, sel, stt))
    check_rc(L.arbor_compact(kv, k, sel, stt, workspace(kv)))
    torch.cuda.synchronize()
    return sel.cpu().numpy(), int(stt)


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("mode", [0, 1])
def test_select_compact_bit_exact(seed, mode):
    st = rand_tree_state(seed, V=30, max_n=90, dtype="bf16" if seed % 2 else "f32",
                         d=128 if seed % 2 else 64)
    kv = to_gpu(st)
    ost = oracle_state(st)
    rng = np.random.default_rng(seed + 50)
    p = dict(PARAMS, select_mode=mode)
    for event in range(2):                                  # nested events
        A = rand_A(st["num_tokens"], seed * 10 + event)
        k = np.array([int(rng.integers(0, c + 1)) if rng.random() < 0.7 else c
                      for c in ost["n_kept"]])
        sel_o, so = O.select(ost, A, k, p["l_tail"], mode)
        assert so == O.OK
        sel_g, sg = _event(st, kv, A, k, p)
        assert sg == L.OK
        for i, keep in sel_o.items():
            b = int(ost["tok_off"][i])
            assert sel_g[b:b + len(keep)].tolist() == keep, (event, i)
        ost = O.compact(ost, k, sel_o)
        assert_same_pool(gpu_to_oracle(kv), ost)


def test_select_nan_is_rejected_and_state_unchanged():
    st = rand_tree_state(3, V=12)
    kv = to_gpu(st)
    before = gpu_to_oracle(kv)
    A = rand_A(st["num_tokens"], 0)
    A[int(st["tok_off"][2]) + 1] = np.nan
    k = np.zeros(12, dtype=np.int32)
    sel, sg = _event(st, kv, A, k, PARAMS)
    assert sg == L.ENONFINITE
    assert_same_pool(gpu_to_oracle(kv), before)


def test_compact_rejects_bad_selection():
    st = rand_tree_state(4, V=8, min_n=20)
    kv = to_gpu(st)
    before = gpu_to_oracle(kv)
    N = st["num_tokens"]
    k = torch.tensor([3] * 8, dtype=torch.int32, device="cuda")
    sel = torch.zeros(N, dtype=torch.int32, device="cuda")      # [0, 0, 0]: not increasing
    stt = status()
    check_rc(L.arbor_compact(kv, k, sel, stt, workspace(kv)))
    torch.cuda.synchronize()
    assert int(stt) == L.EINVAL
    assert_same_pool(gpu_to_oracle(kv), before)


# --------------------------------------------------------------------------- rehydrate
@pytest.mark.parametrize("seed", range(4))
def test_rehydrate_bit_exact_and_restores_full_retention(seed):
    st = rand_tree_state(seed, V=25, max_n=80, dtype="bf16")
    kv = to_gpu(st)
    ost = oracle_state(st)
    pristine = gpu_to_oracle(kv)
    rng = np.random.default_rng(seed)
    A = rand_A(st["num_tokens"], seed)
    k = np.array([int(rng.integers(0, c + 1)) for c in ost["n_kept"]])
    sel_o, _ = O.select(ost, A, k, 5)
    ost = O.compact(ost, k, sel_o)
    _event(st, kv, A, k, PARAMS)
    on_path = (rng.random(25) < 0.6).astype(np.uint8)
    ost, so = O.rehydrate(ost, on_path, np_float(st["host_k"]), np_float(st["host_v"]))
    stt = status()
    hk = st["host_k"].pin_memory()
    hv = st["host_v"].pin_memory()
    check_rc(L.arbor_rehydrate(kv, torch.tensor(on_path, device="cuda"), hk, hv, stt,
                               workspace(kv)))
    torch.cuda.synchronize()
    assert int(stt) == so == L.OK
    got = gpu_to_oracle(kv)
    assert_same_pool(got, ost)
    # rehydrated nodes hold exactly the never-evicted bytes
    for i in np.nonzero(on_path)[0]:
        assert int(got["n_kept"][i]) == int(got["n_full"][i])
    full_on = np.ones(25, np.uint8)
    ost2, _ = O.rehydrate(ost, full_on, np_float(st["host_k"]), np_float(st["host_v"]))
    check_rc(L.arbor_rehydrate(kv, torch.tensor(full_on, device="cuda"), hk, hv, stt,
                               workspace(kv)))
    torch.cuda.synchronize()
    got = gpu_to_oracle(kv)
    assert_same_pool(got, ost2)
    for i in range(25):
        po = int(got["page_off"][i])
        po0 = int(pristine["page_off"][i])
        for s in range(int(got["n_full"][i])):
            pg, pg0 = int(got["page_table"][po + s // 16]), int(pristine["page_table"][po0 + s // 16])
            assert np.array_equal(got["k"][:, pg, :, s % 16].view(np.uint32),
                                  pristine["k"][:, pg0, :, s % 16].view(np.uint32))


def test_rehydrate_out_of_pages_changes_nothing():
    st = rand_tree_state(5, V=10, min_n=20, spare=0)
    kv = to_gpu(st)
    A = rand_A(st["num_tokens"], 1)
    _event(st, kv, A, np.zeros(10, np.int32), PARAMS)
    kv.free_top.fill_(1)
    before = gpu_to_oracle(kv)
    stt = status()
    check_rc(L.arbor_rehydrate(kv, torch.ones(10, dtype=torch.uint8, device="cuda"),
                               st["host_k"].pin_memory(), st["host_v"].pin_memory(), stt,
                               workspace(kv)))
    torch.cuda.synchronize()
    assert int(stt) == L.ENOPAGES
    assert_same_pool(gpu_to_oracle(kv), before)


# --------------------------------------------------------------------------- score
def _gpu_score(st, kv, p, A0=None, rows0=None, observers=None, q_win=None):
    V = kv.num_nodes
    obs = st["observers"] if observers is None else observers
    q = st["q_win"] if q_win is None else q_win
    A = (torch.zeros(st["num_tokens"]) if A0 is None else torch.tensor(A0)).cuda()
    rows = (torch.zeros(V, dtype=torch.int64) if rows0 is None else torch.tensor(rows0)).cuda()
    a = torch.empty(V, device="cuda")
    s = torch.empty(V, device="cuda")
    stt = status()
    ws = workspace(kv, max_observers=obs.numel(), window=st["window"],
                   n_slice=len(st["slice_layers"]))
    check_rc(L.arbor_score(kv, obs.cuda(), q.cuda().contiguous(), st["window"], st["slice_layers"],
                           st["v_sig"].cuda(), st["u_sig"].cuda(), A, rows, a, s, p, stt, ws))
    torch.cuda.synchronize()
    return A.cpu().numpy(), rows.cpu().numpy(), a.cpu().numpy(), s.cpu().numpy(), int(stt)


def _close(g, o, rel=1e-4, atol=1e-30):
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    bad = np.abs(g - o) > rel * np.abs(o) + atol
    assert not bad.any(), (np.nonzero(bad)[0][:10], g[bad][:5], o[bad][:5])


def _oracle_score(st, ost, p, A0=None, rows0=None):
    V = len(ost["parent"])
    return O.score(ost, st["observers"].tolist(), np_float(st["q_win"]), st["window"],
                   st["slice_layers"], st["q_per_kv"], st["v_sig"].numpy(), st["u_sig"].numpy(),
                   np.zeros(st["num_tokens"], np.float32) if A0 is None else A0,
                   np.zeros(V, np.int64) if rows0 is None else rows0,
                   theta=p["theta"], self_window=p["score_self_window"])


def test_score_tiny_config():
    st = synth.build_config("tiny")
    kv = to_gpu(st)
    ost = oracle_state(st)
    p = st["params"]
    A, rows, a, s, sg = _gpu_score(st, kv, p)
    Ao, ro, ao, so = _oracle_score(st, ost, p)
    assert sg == L.OK
    _close(A, Ao)
    assert np.array_equal(rows, ro)
    _close(a, ao)
    _close(s, so)


@pytest.mark.parametrize("seed,self_window,dtype", [(0, 0, "bf16"), (1, 1, "bf16"),
                                                    (2, 0, "f32"), (3, 1, "f32")])
def test_score_random_trees(seed, self_window, dtype):
    st = rand_tree_state(seed, V=14, max_n=75, min_n=2, G=4 if dtype == "bf16" else 1,
                         d=128 if dtype == "bf16" else 64, dtype=dtype, window=12)
    kv = to_gpu(st)
    ost = oracle_state(st)
    p = dict(PARAMS, score_self_window=self_window, theta=(0.5, -1.0, 2.0))
    A0 = (np.random.default_rng(seed).random(st["num_tokens"]) * 3).astype(np.float32)
    r0 = np.arange(14, dtype=np.int64)
    A, rows, a, s, sg = _gpu_score(st, kv, p, A0, r0)
    Ao, ro, ao, so = _oracle_score(st, ost, p, A0, r0)
    assert sg == L.OK
    _close(A, Ao)
    assert np.array_equal(rows, ro)
    _close(a, ao)
    _close(s, so)
    # bitwise reproducible
    A2, *_ = _gpu_score(st, kv, p, A0, r0)
    assert np.array_equal(A.view(np.uint32), A2.view(np.uint32))


# rows per (observer, slice layer, kv head) = G * W; a row group holds 64 rows
# (bf16) or 32 (fp32), and a workgroup covers 2 or 4 groups that share its key
# tiles: 3 and 5 groups leave empty groups in the last workgroup, and chains of
# one to a few sub-pages give key splits with a step fewer than the others
@pytest.mark.parametrize("seed,dtype,d,G,W", [(20, "bf16", 128, 4, 32),    # 2 groups
                                              (21, "bf16", 128, 4, 40),    # 3 groups
                                              (22, "bf16", 64, 8, 32),     # 4 groups
                                              (23, "bf16", 128, 8, 36),    # 5 groups
                                              (24, "f32", 64, 4, 20),      # 3 groups
                                              (25, "f32", 128, 4, 40)])    # 5 groups
def test_score_shared_key_tiles(seed, dtype, d, G, W):
    st = rand_tree_state(seed, V=16, max_n=90, min_n=1, G=G, d=d, dtype=dtype, window=W)
    kv = to_gpu(st)
    ost = oracle_state(st)
    p = dict(PARAMS, score_self_window=seed % 2, theta=(0.5, -1.0, 2.0))
    A0 = (np.random.default_rng(seed).random(st["num_tokens"]) * 3).astype(np.float32)
    r0 = np.arange(16, dtype=np.int64)
    A, rows, a, s, sg = _gpu_score(st, kv, p, A0, r0)
    Ao, ro, ao, so = _oracle_score(st, ost, p, A0, r0)
    assert sg == L.OK
    _close(A, Ao)
    assert np.array_equal(rows, ro)
    _close(a, ao)
    _close(s, so)
    A2, *_ = _gpu_score(st, kv, p, A0, r0)
    assert np.array_equal(A.view(np.uint32), A2.view(np.uint32))


@pytest.mark.parametrize("dtype,d,G", [("bf16", 128, 4), ("bf16", 128, 8), ("f32", 64, 2)])
def test_score_shared_key_tiles_long_chain(dtype, d, G):
    """Chains of more than 64 steps per key split: the sub-page table is read
    in windows of 64 steps, and the waves sharing the tiles meet at the end
    of each window before the ring is reused."""
    parent, n_full = [-1, 0, 1], [2500, 1700, 300]
    st = synth.build_state(parent, n_full, layers=2, kv_heads=2, q_per_kv=G, head_dim=d,
                           dtype=dtype, seed=31, shuffle_pages=True, page_size=16, window=32,
                           active=[2], heavy_frac=0.01)
    kv = to_gpu(st)
    ost = oracle_state(st)
    p = dict(PARAMS, score_self_window=1 if G == 8 else 0)
    A, rows, a, s, sg = _gpu_score(st, kv, p)
    Ao, ro, ao, so = _oracle_score(st, ost, p)
    assert sg == L.OK
    _close(A, Ao)
    assert np.array_equal(rows, ro)
    _close(s, so)


def test_score_after_eviction():
    st = rand_tree_state(7, V=12, max_n=60, min_n=10, G=4, window=16)
    kv = to_gpu(st)
    ost = oracle_state(st)
    rng = np.random.default_rng(0)
    A = rand_A(st["num_tokens"], 3, ties=False)
    k = np.array([int(rng.integers(1, c + 1)) for c in ost["n_kept"]])
    sel_o, _ = O.select(ost, A, k, 5)
    ost = O.compact(ost, k, sel_o)
    _event(st, kv, A, k, PARAMS)
    A, rows, a, s, sg = _gpu_score(st, kv, PARAMS)
    Ao, ro, ao, so = _oracle_score(st, ost, PARAMS)
    _close(A, Ao)
    assert np.array_equal(rows, ro)
    _close(s, so)


def test_score_long_chain():
    """Chains longer than the score kernel's in-LDS sub-page table."""
    parent, n_full = [-1, 0, 1], [7000, 6000, 5003]
    st = synth.build_state(parent, n_full, layers=1, kv_heads=1, q_per_kv=1, head_dim=64,
                           dtype="bf16", seed=3, shuffle_pages=True, page_size=32, window=4,
                           active=[2], heavy_frac=0.01)
    kv = to_gpu(st)
    ost = oracle_state(st)
    A, rows, a, s, sg = _gpu_score(st, kv, PARAMS)
    Ao, ro, ao, so = _oracle_score(st, ost, PARAMS)
    assert sg == L.OK
    _close(A, Ao)
    assert np.array_equal(rows, ro)
    _close(s, so)


# --------------------------------------------------------------------------- decode
def _gpu_decode(st, kv, leaves, l0, l1, q, out_dtype=torch.float32):
    n = leaves.numel()
    Hq = kv.kv_heads * kv.q_per_kv
    out = torch.empty((n, l1 - l0, Hq, kv.head_dim), dtype=out_dtype, device="cuda")
    lse = torch.empty((n, l1 - l0, Hq), device="cuda")
    stt = status()
    ws = workspace(kv, max_leaves=n, max_layers=l1 - l0)
    check_rc(L.arbor_tree_decode_attn(kv, leaves.cuda(), l0, l1, q.cuda().contiguous(), out, lse,
                                      0.0, stt, ws))
    torch.cuda.synchronize()
    return out.float().cpu().numpy(), lse.cpu().numpy(), int(stt)


def _bf16_round(x):
    return torch.tensor(x, dtype=torch.float64).to(torch.bfloat16).double().numpy()


@pytest.mark.parametrize("seed,dtype,G,leaves", [(0, "bf16", 4, None), (1, "bf16", 8, None),
                                                 (2, "f32", 1, None), (3, "bf16", 4, "many")])
def test_decode_random_trees(seed, dtype, G, leaves):
    V = 40
    act = None
    if leaves == "many":
        parent, _ = synth.random_tree(V, 5, seed, min_tokens=1)
        act = [i for i in range(V) if i not in parent][:14]     # > 64 rows at the root
    st = rand_tree_state(seed, V=V, max_n=700 if seed == 1 else 90, min_n=1, G=G,
                         d=128 if dtype == "bf16" else 64, dtype=dtype, active=act, L_=3)
    kv = to_gpu(st)
    ost = oracle_state(st)
    rng = np.random.default_rng(seed)
    if seed % 2 == 0:                                  # decode over an evicted state too
        A = rand_A(st["num_tokens"], seed, ties=False)
        k = np.array([int(rng.integers(0, c + 1)) for c in ost["n_kept"]])
        sel_o, _ = O.select(ost, A, k, 5)
        ost = O.compact(ost, k, sel_o)
        _event(st, kv, A, k, PARAMS)
    leaves_t = st["active"]
    q = st["q_dec"][:, 1:3]
    o_o, lse_o = O.tree_decode_attn(ost, leaves_t.tolist(), 1, 3, np_float(q), G)
    out, lse, sg = _gpu_decode(st, kv, leaves_t, 1, 3, q)
    assert sg == L.OK
    assert np.max(np.abs(out - o_o)) <= 2e-3
    fin = np.isfinite(lse_o)
    assert np.max(np.abs(lse[fin] - lse_o[fin])) <= 1e-4 * max(1.0, np.abs(lse_o[fin]).max())
    if dtype == "bf16":
        outb, _, _ = _gpu_decode(st, kv, leaves_t, 1, 3, q, torch.bfloat16)
        ref = _bf16_round(o_o)
        ulp = np.abs(ref) * 2.0 ** -7
        assert np.all(np.abs(outb - ref) <= np.maximum(2e-3, ulp) + 1e-12)
    out2, _, _ = _gpu_decode(st, kv, leaves_t, 1, 3, q)
    assert np.array_equal(out.view(np.uint32), out2.view(np.uint32))


def test_decode_after_rehydrate_equals_never_evicted():
    st = rand_tree_state(11, V=20, max_n=120, min_n=30, G=4)
    kv = to_gpu(st)
    q = st["q_dec"]
    ref, ref_lse, _ = _gpu_decode(st, kv, st["active"], 0, 2, q)
    A = rand_A(st["num_tokens"], 2, ties=False)
    _event(st, kv, A, np.array([3] * 20, np.int32), PARAMS)
    check_rc(L.arbor_rehydrate(kv, torch.ones(20, dtype=torch.uint8, device="cuda"),
                               st["host_k"].pin_memory(), st["host_v"].pin_memory(), status(),
                               workspace(kv)))
    out, lse, _ = _gpu_decode(st, kv, st["active"], 0, 2, q)
    assert np.array_equal(out.view(np.uint32), ref.view(np.uint32))
