"""The eviction event (score, allocate, select, compact, tree decode) captured as
a HIP graph and replayed: every replay must equal the eager run bitwise, with
eager work and synchronisations between the replays (bench.py times the
replayed graph)."""
import numpy as np
import pytest
import torch

from paper_2605_22106_amd import _lib as L
from paper_2605_22106_amd import synth
from tests.gpu_helpers import check_rc

pytestmark = pytest.mark.gpu


def test_graph_replay_equals_eager():
    parent, n_full = synth.random_tree(40, 90, seed=7, min_tokens=20)
    leaves = [i for i in range(40) if i not in parent]
    st = synth.build_state(parent, n_full, layers=3, kv_heads=2, q_per_kv=4, head_dim=128,
                           dtype="bf16", seed=7, shuffle_pages=True, window=16,
                           active=leaves[:3], heavy_frac=0.05)
    kv = L.kv_state_from(st, "cuda")
    pristine = kv.clone()
    V, N = kv.num_nodes, kv.num_tokens
    dev = "cuda"
    p = dict(alpha_max=float("inf"), gamma=2.0, lambda_d=0.1, lambda_delta=0.5, eta=0.8,
             r_min=0.05, k_min=4, l_tail=6, theta=(1.0, 1.0, 1.0), select_mode=0,
             score_self_window=0)
    obs = st["observers"].to(dev)
    q_win = st["q_win"].to(dev).contiguous()
    q_dec = st["q_dec"].to(dev).contiguous()
    v_sig, u_sig = st["v_sig"].to(dev), st["u_sig"].to(dev)
    active = st["active"].to(dev)
    budget = int(0.4 * N)
    A = torch.zeros(N, device=dev)
    rows = torch.zeros(V, dtype=torch.int64, device=dev)
    a, s = torch.empty(V, device=dev), torch.empty(V, device=dev)
    k = torch.empty(V, dtype=torch.int32, device=dev)
    delta = torch.empty_like(k)
    on_path = torch.empty(V, dtype=torch.uint8, device=dev)
    sel = torch.full((N,), -1, dtype=torch.int32, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    Hq = kv.kv_heads * kv.q_per_kv
    out = torch.empty((active.numel(), kv.layers, Hq, kv.head_dim), device=dev)
    lse = torch.empty((active.numel(), kv.layers, Hq), device=dev)
    ws = torch.empty(L.arbor_workspace_size(kv, max_observers=V, window=16, n_slice=2,
                                            max_leaves=8, max_layers=kv.layers),
                     dtype=torch.uint8, device=dev)

    def event():
        check_rc(L.arbor_score(kv, obs, q_win, 16, st["slice_layers"], v_sig, u_sig, A, rows, a,
                               s, p, status, ws))
        check_rc(L.arbor_allocate(kv, active, budget, s, p, k, delta, on_path, status, ws))
        check_rc(L.arbor_select(kv, A, k, p, sel, status))
        check_rc(L.arbor_compact(kv, k, sel, status, ws))
        check_rc(L.arbor_tree_decode_attn(kv, active, 0, kv.layers, q_dec, out, lse, 0.0, status,
                                          ws))

    def reset():
        kv.copy_from(pristine)
        A.zero_()
        rows.zero_()
        status.zero_()

    def snapshot():
        torch.cuda.synchronize()
        return [t.detach().clone() for t in (A, rows, a, s, k, kv.n_kept, kv.page_table,
                                             kv.slot_pos, kv.free_stack, kv.free_top, out, lse,
                                             status)] + [kv.k.clone(), kv.v.clone()]

    reset()
    event()
    eager = snapshot()
    assert int(status) >= 0
    assert int((kv.n_kept < pristine.n_kept).sum()) > 0, "the budget must evict something"

    reset()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        event()
    torch.cuda.synchronize()
    other = torch.zeros(N, device=dev)
    for rep in range(3):
        reset()
        torch.cuda.synchronize()
        g.replay()
        got = snapshot()
        for x, y in zip(eager, got):
            assert torch.equal(x.view(torch.uint8) if x.dtype == torch.bfloat16 else x,
                               y.view(torch.uint8) if y.dtype == torch.bfloat16 else y), rep
        # eager work between the replays, on other buffers
        other.zero_()
        check_rc(L.arbor_score(kv, obs, q_win, 16, st["slice_layers"], v_sig, u_sig, other,
                               torch.zeros(V, dtype=torch.int64, device=dev), a.clone(),
                               s.clone(), p, torch.zeros(1, dtype=torch.int32, device=dev), ws))
        torch.cuda.synchronize()
