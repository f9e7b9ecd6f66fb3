"""GPU parity of arbor_tree_decode_attn_scored: the decode outputs equal the
plain decode bitwise, and A / rows_seen equal the oracle's decode-time credit
(|g - o| <= 1e-4 |o| + 1e-30 on A, bit-exact rows_seen)."""
import numpy as np
import pytest
import torch

from oracle import arbor_oracle as O
from paper_2605_22106_amd import _lib as L
from paper_2605_22106_amd import synth
from tests.gpu_helpers import check_rc, gpu_to_oracle, status, to_gpu, workspace
from tests.helpers import np_float, oracle_state
from tests.test_gpu_parity import PARAMS, _close, _event, _gpu_decode, rand_A, rand_tree_state

pytestmark = pytest.mark.gpu


def _scored(st, kv, leaves, l0, l1, q, slice_layers, self_window, A0, r0, out_dtype=torch.float32):
    n = leaves.numel()
    Hq = kv.kv_heads * kv.q_per_kv
    out = torch.empty((n, l1 - l0, Hq, kv.head_dim), dtype=out_dtype, device="cuda")
    lse = torch.empty((n, l1 - l0, Hq), device="cuda")
    A = torch.tensor(A0, device="cuda")
    rows = torch.tensor(r0, device="cuda")
    stt = status()
    ws = workspace(kv, max_leaves=max(n, 1), max_layers=l1 - l0, n_slice=len(slice_layers))
    check_rc(L.arbor_tree_decode_attn_scored(kv, leaves.cuda(), l0, l1, q.cuda().contiguous(),
                                             out, lse, 0.0, slice_layers, self_window, A, rows,
                                             stt, ws))
    torch.cuda.synchronize()
    return (out.float().cpu().numpy(), lse.cpu().numpy(), A.cpu().numpy(), rows.cpu().numpy(),
            int(stt))


def _check(st, kv, ost, leaves, l0, l1, q, S, sw, seed):
    rng = np.random.default_rng(seed)
    A0 = (rng.random(st["num_tokens"]) * 2).astype(np.float32)
    r0 = rng.integers(0, 100, size=kv.num_nodes).astype(np.int64)
    lt = torch.tensor(leaves, dtype=torch.int32)
    out, lse, A, rows, sg = _scored(st, kv, lt, l0, l1, q, S, sw, A0, r0)
    assert sg == L.OK
    out_p, lse_p, sp = _gpu_decode(st, kv, lt, l0, l1, q)
    assert sp == L.OK
    assert np.array_equal(out.view(np.uint32), out_p.view(np.uint32))
    assert np.array_equal(lse.view(np.uint32), lse_p.view(np.uint32))
    Ao, ro = O.decode_credit(ost, leaves, l0, np_float(q), st["q_per_kv"], S, A0, r0,
                             self_window=sw)
    _close(A, Ao)
    assert np.array_equal(rows, ro)
    _, _, A2, rows2, _ = _scored(st, kv, lt, l0, l1, q, S, sw, A0, r0)
    assert np.array_equal(A.view(np.uint32), A2.view(np.uint32))    # reproducible
    assert np.array_equal(rows, rows2)
    return A, A0


@pytest.mark.parametrize("seed,dtype,G,sw", [(0, "bf16", 4, 0), (1, "bf16", 8, 1),
                                             (2, "f32", 1, 0), (3, "f32", 2, 1)])
def test_scored_decode_random_trees(seed, dtype, G, sw):
    st = rand_tree_state(seed, V=30, max_n=300 if seed == 1 else 90, min_n=1, G=G,
                         d=128 if dtype == "bf16" else 64, dtype=dtype, L_=4)
    kv = to_gpu(st)
    ost = oracle_state(st)
    if seed % 2 == 0:                                  # an evicted state too
        rng = np.random.default_rng(seed)
        A = rand_A(st["num_tokens"], seed, ties=False)
        k = np.array([int(rng.integers(0, c + 1)) for c in ost["n_kept"]])
        sel_o, _ = O.select(ost, A, k, 5)
        ost = O.compact(ost, k, sel_o)
        _event(st, kv, A, k, PARAMS)
    leaves = st["active"].tolist()
    q = st["q_dec"][:, 1:4]
    _check(st, kv, ost, leaves, 1, 4, q, [2, 3], sw, seed)


@pytest.mark.parametrize("sw", [0, 1])
def test_scored_decode_many_leaves_share_ancestors(sw):
    """Fourteen leaves of a bushy tree: more than 16 query rows per kv head
    on the shared ancestors (several row blocks per key tile), one leaf
    listed twice, one leaf an ancestor of another listed leaf."""
    V = 40
    parent, _ = synth.random_tree(V, 5, 3, min_tokens=1)
    lv = [i for i in range(V) if i not in parent][:13]
    lv = lv + [lv[0], parent[lv[5]]]
    st = rand_tree_state(3, V=V, max_n=90, min_n=1, G=4, active=lv, L_=2)
    kv = to_gpu(st)
    ost = oracle_state(st)
    _check(st, kv, ost, lv, 0, 2, st["q_dec"], [1, 0, 1], sw, 3)


def test_scored_decode_empty_chain_and_single_layer():
    """A leaf whose chain holds no resident token gets rows counted and gives
    nothing; slice of one layer; a one-token root."""
    parent, n_full = [-1, 0, 0, 1, 2], [1, 20, 33, 17, 9]
    st = synth.build_state(parent, n_full, layers=3, kv_heads=2, q_per_kv=4, head_dim=128,
                           dtype="bf16", seed=9, page_size=16, active=[3, 4],
                           shuffle_pages=True)
    kv = to_gpu(st)
    ost = oracle_state(st)
    A = rand_A(st["num_tokens"], 9, ties=False)
    k = np.array([0, 0, 5, 0, 9], np.int32)          # chain of leaf 3 emptied
    sel_o, _ = O.select(ost, A, k, 5)
    ost = O.compact(ost, k, sel_o)
    _, sg = _event(st, kv, A, k, PARAMS)
    assert sg == L.OK
    Ag, A0 = _check(st, kv, ost, [3, 4], 0, 3, st["q_dec"], [2], 0, 9)
    assert np.array_equal(Ag[:1 + 20], A0[:1 + 20])   # root and node 1 hold nothing


def test_scored_decode_rejects_bad_slices():
    st = rand_tree_state(5, V=8, max_n=20, G=2, L_=3)
    kv = to_gpu(st)
    lt = st["active"]
    Hq = kv.kv_heads * kv.q_per_kv
    out = torch.empty((lt.numel(), 2, Hq, kv.head_dim), device="cuda")
    A = torch.zeros(st["num_tokens"], device="cuda")
    rows = torch.zeros(kv.num_nodes, dtype=torch.int64, device="cuda")
    ws = workspace(kv, max_leaves=lt.numel(), max_layers=2, n_slice=8)
    q = st["q_dec"][:, 1:3].cuda().contiguous()
    for sl, sw in (([0], 0), ([3], 0), ([], 0), ([1] * 9, 0), ([1], 2)):
        rc = L.arbor_tree_decode_attn_scored(kv, lt.cuda(), 1, 3, q, out, None, 0.0, sl, sw, A,
                                             rows, status(), ws)
        assert rc == L.EINVAL, (sl, sw)


def test_incremental_scores_drive_an_eviction():
    """A kept up to date by three scored decode steps (new queries each step)
    matches the oracle's running credit, and an eviction driven by it selects
    the same tokens on both sides (the GPU's A handed to both)."""
    st = rand_tree_state(21, V=20, max_n=120, min_n=20, G=4, L_=2)
    kv = to_gpu(st)
    ost = oracle_state(st)
    N, V = st["num_tokens"], kv.num_nodes
    Hq = kv.kv_heads * kv.q_per_kv
    leaves = st["active"].tolist()
    lt = st["active"].cuda()
    A_o = np.zeros(N, np.float32)
    r_o = np.zeros(V, np.int64)
    A_g = torch.zeros(N, device="cuda")
    r_g = torch.zeros(V, dtype=torch.int64, device="cuda")
    ws = workspace(kv, max_leaves=len(leaves), max_layers=2, n_slice=1)
    gen = torch.Generator().manual_seed(21)
    for step in range(3):
        q = torch.randn((len(leaves), 2, Hq, kv.head_dim), generator=gen).to(torch.bfloat16)
        out = torch.empty((len(leaves), 2, Hq, kv.head_dim), device="cuda")
        stt = status()
        check_rc(L.arbor_tree_decode_attn_scored(kv, lt, 0, 2, q.cuda().contiguous(), out, None,
                                                 0.0, [1], 0, A_g, r_g, stt, ws))
        torch.cuda.synchronize()
        assert int(stt) == L.OK
        A_o, r_o = O.decode_credit(ost, leaves, 0, np_float(q), kv.q_per_kv, [1], A_o, r_o)
    _close(A_g.cpu().numpy(), A_o)
    assert np.array_equal(r_g.cpu().numpy(), r_o)
    A = A_g.cpu().numpy()
    rng = np.random.default_rng(21)
    k = np.array([int(rng.integers(1, c + 1)) for c in ost["n_kept"]], np.int32)
    sel_o, _ = O.select(ost, A, k, PARAMS["l_tail"])
    sel, sg = _event(st, kv, A, k, PARAMS)
    assert sg == L.OK
    for i, keep in sel_o.items():
        b = int(ost["tok_off"][i])
        assert np.array_equal(sel[b:b + len(keep)], np.array(keep, np.int32)), i
