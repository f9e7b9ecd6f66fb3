"""GPU parity at the benchmark's full sizes, in the launch configuration
bench.py times (same entry points, same workspace sizing, same inputs).

The oracle cannot replay a whole 32-layer pool in fp64 in test time, so each
stage is checked on what it can compute exactly at this size:

* score: every observer of the llama8b tree, against the oracle run on the
  two slice layers only (the only K the definition reads); the 70B-shaped tree
  on a sample of observers (the observer list is an input of both sides);
* allocate / select: bit-exact on the whole tree, fed the GPU's s and A;
* compact: page tables, slot maps, resident counts and free stack bit-exact
  against the oracle run on the metadata; K/V bytes of sampled moved rows, in
  every layer and kv head, equal the pristine rows of their positions;
* decode: sampled (leaf, layer, query head) outputs against an fp64 softmax
  over the chain's rows read back from the pool;
* rehydrate: every restored Path* row equals the pristine row bitwise, and the
  page count is conserved.
"""
import math

import numpy as np
import pytest
import torch

from oracle import arbor_oracle as O
from paper_2605_22106_amd import _lib as L
from paper_2605_22106_amd import synth
from tests.gpu_helpers import check_rc, status
from tests.helpers import np_float

pytestmark = pytest.mark.gpu


def _meta(kv, k=None, v=None):
    """Oracle state with the pool metadata; K/V only where a check needs them."""
    d = {key: getattr(kv, key).cpu().numpy().astype(np.int64) for key in
         ("parent", "n_full", "tok_off", "page_off", "n_kept", "page_table", "slot_pos",
          "free_stack")}
    d["free_top"] = np.int64(int(kv.free_top.reshape(-1)[0]))
    d["page_size"] = kv.page_size
    P = kv.page_size
    npages = kv.slot_pos.shape[0]
    d["k"] = np.zeros((1, npages, 1, P, 1), np.float32) if k is None else k
    d["v"] = np.zeros((1, npages, 1, P, 1), np.float32) if v is None else v
    return d


def _workspace(kv, st, n_obs):
    chain_max = max(sum(int(st["n_full"][a]) for a in O.chain(st["parent"].tolist(), j))
                    for j in range(kv.num_nodes))
    n = L.arbor_workspace_size(kv, max_context=chain_max, max_observers=n_obs,
                               window=st["window"], n_slice=len(st["slice_layers"]),
                               max_leaves=64, max_layers=kv.layers)
    return torch.empty(n, dtype=torch.uint8, device="cuda")


def _gpu_score(kv, st, obs, q_win, p, ws):
    V, N = kv.num_nodes, kv.num_tokens
    A = torch.zeros(N, device="cuda")
    rows = torch.zeros(V, dtype=torch.int64, device="cuda")
    a = torch.empty(V, device="cuda")
    s = torch.empty(V, device="cuda")
    stt = status()
    check_rc(L.arbor_score(kv, obs, q_win, st["window"], st["slice_layers"], st["v_sig"].cuda(),
                           st["u_sig"].cuda(), A, rows, a, s, p, stt, ws))
    torch.cuda.synchronize()
    assert int(stt) == L.OK
    return A, rows, a, s


def _oracle_score(kv, st, obs_list, q_np, p):
    """The oracle on the slice layers only (K of other layers is never read)."""
    sl = st["slice_layers"]
    ksl = kv.k[sl].float().cpu().numpy()
    ost = _meta(kv, k=ksl)
    V = kv.num_nodes
    return O.score(ost, obs_list, q_np, st["window"], list(range(len(sl))), st["q_per_kv"],
                   st["v_sig"].numpy(), st["u_sig"].numpy(), np.zeros(kv.num_tokens, np.float32),
                   np.zeros(V, np.int64), theta=p["theta"], self_window=p["score_self_window"])


def _close(g, o, rel=1e-4, atol=1e-30):
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    bad = np.abs(g - o) > rel * np.abs(o) + atol
    assert not bad.any(), (np.nonzero(bad)[0][:10], g[bad][:5], o[bad][:5])


def _rows(kv, pool, pages, rs, layer=None):
    """K or V rows [n, L, Hkv, d] of (page, r) slots, as a CPU tensor."""
    x = pool[:, pages, :, rs, :] if layer is None else pool[layer][pages, :, rs, :]
    return x.cpu()


def _decode_layers_vs_oracle(kv, st, out_np, q, layers):
    """out_np[:, l] for every active leaf and query head of each layer l against
    O.tree_decode_attn run on that layer of the current pool (fp64)."""
    leaves = st["active"].tolist()
    for l in layers:
        ost = _meta(kv, k=kv.k[l:l + 1].float().cpu().numpy(),
                    v=kv.v[l:l + 1].float().cpu().numpy())
        o_o, _ = O.tree_decode_attn(ost, leaves, 0, 1, np_float(q[:, l:l + 1]), kv.q_per_kv)
        err = np.abs(out_np[:, l:l + 1] - o_o).max()
        assert err <= 2e-3, (l, err)


@pytest.fixture(scope="module")
def llama8b():
    cfg = synth.CONFIGS["llama8b"]
    st = synth.build_config(cfg, device="cuda")
    kv = L.kv_state_from(st, "cuda")
    return st, kv, kv.clone()


def test_llama8b_event_stage_by_stage(llama8b):
    st, kv, pristine = llama8b
    kv.copy_from(pristine)
    p = st["params"]
    V, N, P = kv.num_nodes, kv.num_tokens, kv.page_size
    obs = st["observers"].cuda()
    ws = _workspace(kv, st, obs.numel())
    q_win = st["q_win"].cuda().contiguous()

    # score: every observer, against the oracle on the slice layers
    A, rows, a, s = _gpu_score(kv, st, obs, q_win, p, ws)
    Ao, ro, ao, so = _oracle_score(kv, st, st["observers"].tolist(), np_float(st["q_win"]), p)
    _close(A.cpu().numpy(), Ao)
    assert np.array_equal(rows.cpu().numpy(), ro)
    _close(a.cpu().numpy(), ao)
    _close(s.cpu().numpy(), so)

    # allocate: the GPU's s on both sides
    active = st["active"].cuda()
    k = torch.empty(V, dtype=torch.int32, device="cuda")
    delta = torch.empty_like(k)
    on_path = torch.empty(V, dtype=torch.uint8, device="cuda")
    stt = status()
    check_rc(L.arbor_allocate(kv, active, st["budget"], s, p, k, delta, on_path, stt, ws))
    torch.cuda.synchronize()
    s_np = s.cpu().numpy()
    meta0 = _meta(kv)
    ko, do, po, so_ = O.allocate(meta0["parent"], meta0["n_full"], meta0["n_kept"],
                                 st["active"].tolist(), st["budget"], s_np, p)
    assert int(stt) == so_
    assert np.array_equal(k.cpu().numpy(), ko)
    assert np.array_equal(delta.cpu().numpy(), do)
    assert np.array_equal(on_path.cpu().numpy().astype(bool), po.astype(bool))

    # select: the GPU's A on both sides
    sel = torch.full((N,), -7, dtype=torch.int32, device="cuda")
    check_rc(L.arbor_select(kv, A, k, p, sel, stt))
    torch.cuda.synchronize()
    sel_o, sst = O.select(meta0, A.cpu().numpy(), ko, p["l_tail"], p["select_mode"])
    assert sst == O.OK and int(stt) == L.OK
    sel_np = sel.cpu().numpy()
    tok_off = meta0["tok_off"]
    for i, keep in sel_o.items():
        b = int(tok_off[i])
        assert np.array_equal(sel_np[b:b + len(keep)], np.array(keep, np.int32)), i

    # compact: metadata bit-exact, sampled moved rows bitwise in every layer/head
    check_rc(L.arbor_compact(kv, k, sel, stt, ws))
    torch.cuda.synchronize()
    assert int(stt) == L.OK
    new_o = O.compact(meta0, ko, sel_o)
    meta1 = _meta(kv)
    for key in ("n_kept", "page_table", "slot_pos"):
        assert np.array_equal(meta1[key], new_o[key]), key
    top = int(meta1["free_top"])
    assert top == int(new_o["free_top"])
    assert np.array_equal(meta1["free_stack"][:top], new_o["free_stack"][:top])
    used = sum(-(-int(c) // P) for c in meta1["n_kept"])
    assert used + top == kv.slot_pos.shape[0]                       # no page lost or doubled
    rng = np.random.default_rng(0)
    moved = [(i, s_) for i, keep in sel_o.items() for s_, pos in enumerate(keep) if pos != s_]
    assert moved, "the event moves rows"
    pick = [moved[j] for j in rng.choice(len(moved), size=min(256, len(moved)), replace=False)]
    pt0 = pristine.page_table.cpu().numpy()
    po_ = meta0["page_off"]
    dst_pages = torch.tensor([int(meta1["page_table"][po_[i] + s_ // P]) for i, s_ in pick])
    dst_r = torch.tensor([s_ % P for _, s_ in pick])
    src_pages = torch.tensor([int(pt0[po_[i] + sel_o[i][s_] // P]) for i, s_ in pick])
    src_r = torch.tensor([sel_o[i][s_] % P for i, s_ in pick])
    for pool_now, pool_then in ((kv.k, pristine.k), (kv.v, pristine.v)):
        got = _rows(kv, pool_now, dst_pages.cuda(), dst_r.cuda())
        want = _rows(kv, pool_then, src_pages.cuda(), src_r.cuda())
        assert torch.equal(got.view(torch.int16), want.view(torch.int16))

    # decode: sampled (leaf, layer, head) against an fp64 softmax over the chain
    Hq = kv.kv_heads * kv.q_per_kv
    q = st["q_dec"].cuda().contiguous()
    nl = active.numel()
    out = torch.empty((nl, kv.layers, Hq, kv.head_dim), device="cuda")
    check_rc(L.arbor_tree_decode_attn(kv, active, 0, kv.layers, q, out, None, 0.0, stt, ws))
    torch.cuda.synchronize()
    assert int(stt) == L.OK
    out_np = out.cpu().numpy()
    scale = 1.0 / math.sqrt(kv.head_dim)
    parent = meta1["parent"].tolist()
    for b, layer, h in zip(rng.integers(0, nl, 48), rng.integers(0, kv.layers, 48),
                           rng.integers(0, Hq, 48)):
        leaf = int(st["active"][b])
        slots = [(int(meta1["page_table"][po_[x] + s_ // P]), s_ % P)
                 for x in O.chain(parent, leaf) for s_ in range(int(meta1["n_kept"][x]))]
        pg = torch.tensor([x for x, _ in slots], device="cuda")
        rr = torch.tensor([r for _, r in slots], device="cuda")
        g = int(h) // kv.q_per_kv
        K = kv.k[int(layer)][pg, g, rr, :].double().cpu().numpy()
        Vv = kv.v[int(layer)][pg, g, rr, :].double().cpu().numpy()
        qv = q[b, int(layer), int(h)].double().cpu().numpy()
        z = scale * (K @ qv)
        w = np.exp(z - z.max())
        o_ref = (w / w.sum()) @ Vv
        err = np.abs(out_np[b, layer, h] - o_ref).max()
        assert err <= 2e-3, (b, layer, h, err)
    # every (leaf, query head) of the two slice layers against the oracle's
    # decode on that layer of the compacted state
    _decode_layers_vs_oracle(kv, st, out_np, q, st["slice_layers"])

    # decode with the decode-time credit: the same outputs bitwise, and A /
    # rows_seen against the oracle on the slice layers (the only K it reads)
    sl = st["slice_layers"]
    A_in = A.clone()
    rows_in = rows.clone()
    out2 = torch.empty_like(out)
    check_rc(L.arbor_tree_decode_attn_scored(kv, active, 0, kv.layers, q, out2, None, 0.0, sl,
                                             0, A, rows, stt, ws))
    torch.cuda.synchronize()
    assert int(stt) == L.OK
    assert torch.equal(out2.view(torch.int32), out.view(torch.int32))
    ost_sl = _meta(kv, k=kv.k[sl].float().cpu().numpy())
    Ao2, ro2 = O.decode_credit(ost_sl, st["active"].tolist(), 0, np_float(q[:, sl]),
                               kv.q_per_kv, list(range(len(sl))), A_in.cpu().numpy(),
                               rows_in.cpu().numpy())
    _close(A.cpu().numpy(), Ao2)
    assert np.array_equal(rows.cpu().numpy(), ro2)

    # rehydrate: move the frontier to other leaves; restored rows are pristine
    leaves = [i for i in range(V) if i not in parent]
    a0 = set(st["active"].tolist())
    alt = [x for x in leaves if x not in a0]
    a1 = torch.tensor([alt[(j * len(alt)) // len(a0) + 3] for j in range(len(a0))],
                      dtype=torch.int32, device="cuda")
    check_rc(L.arbor_allocate(kv, a1, st["budget"], s, p, k, delta, on_path, stt, ws))
    check_rc(L.arbor_rehydrate(kv, on_path, st["host_k"], st["host_v"], stt, ws))
    torch.cuda.synchronize()
    assert int(stt) in (L.OK, L.OVER_BUDGET)
    meta2 = _meta(kv)
    onp = on_path.cpu().numpy().astype(bool)
    restored = [i for i in range(V) if onp[i] and int(meta1["n_kept"][i]) < int(meta2["n_full"][i])]
    assert restored, "the transition re-enters evicted blocks"
    for i in np.nonzero(onp)[0]:
        assert int(meta2["n_kept"][i]) == int(meta2["n_full"][i])
    used = sum(-(-int(c) // P) for c in meta2["n_kept"])
    assert used + int(meta2["free_top"]) == kv.slot_pos.shape[0]
    for i in restored:
        n = int(meta2["n_full"][i])
        pg = torch.tensor([int(meta2["page_table"][po_[i] + s_ // P]) for s_ in range(n)],
                          device="cuda")
        rr = torch.tensor([s_ % P for s_ in range(n)], device="cuda")
        pg0 = torch.tensor([int(pt0[po_[i] + s_ // P]) for s_ in range(n)], device="cuda")
        for pool_now, pool_then in ((kv.k, pristine.k), (kv.v, pristine.v)):
            assert torch.equal(pool_now[:, pg, :, rr, :].view(torch.int16),
                               pool_then[:, pg0, :, rr, :].view(torch.int16)), i


@pytest.fixture(scope="module")
def llama70b():
    cfg = synth.CONFIGS["llama70b"]
    st = synth.build_config(cfg, device="cuda", host_store=False)
    kv = L.kv_state_from(st, "cuda")
    return st, kv


def test_llama70b_score_sample_allocate_select_compact_decode(llama70b):
    """The 70B-shaped tree (80 layers, G = 8, 178K tokens, 58 GB of pool)."""
    st, kv = llama70b
    p = st["params"]
    V, N, P = kv.num_nodes, kv.num_tokens, kv.page_size
    parent = st["parent"].tolist()
    # score on a sample of observers: the root, an inner node, three leaves
    sample = [0, 5, V - 1, V - 100, V - 200]
    obs = torch.tensor(sample, dtype=torch.int32, device="cuda")
    ws = _workspace(kv, st, V)
    idx = [st["observers"].tolist().index(j) for j in sample]
    q_s = st["q_win"][idx].contiguous()
    A, rows, a, s = _gpu_score(kv, st, obs, q_s.cuda(), p, ws)
    Ao, ro, ao, so = _oracle_score(kv, st, sample, np_float(q_s), p)
    _close(A.cpu().numpy(), Ao)
    assert np.array_equal(rows.cpu().numpy(), ro)
    _close(s.cpu().numpy(), so)
    # allocate / select / compact on the whole tree with a synthetic score
    rng = np.random.default_rng(4)
    s_full = torch.tensor(rng.random(V).astype(np.float32), device="cuda")
    A_full = torch.tensor(rng.random(N).astype(np.float32), device="cuda")
    active = st["active"].cuda()
    k = torch.empty(V, dtype=torch.int32, device="cuda")
    delta = torch.empty_like(k)
    on_path = torch.empty(V, dtype=torch.uint8, device="cuda")
    stt = status()
    check_rc(L.arbor_allocate(kv, active, st["budget"], s_full, p, k, delta, on_path, stt, ws))
    sel = torch.full((N,), -7, dtype=torch.int32, device="cuda")
    check_rc(L.arbor_select(kv, A_full, k, p, sel, stt))
    torch.cuda.synchronize()
    meta0 = _meta(kv)
    ko, _, _, so_ = O.allocate(meta0["parent"], meta0["n_full"], meta0["n_kept"],
                               st["active"].tolist(), st["budget"], s_full.cpu().numpy(), p)
    assert np.array_equal(k.cpu().numpy(), ko) and so_ == O.OK
    sel_o, _ = O.select(meta0, A_full.cpu().numpy(), ko, p["l_tail"], p["select_mode"])
    sel_np = sel.cpu().numpy()
    for i, keep in sel_o.items():
        b = int(meta0["tok_off"][i])
        assert np.array_equal(sel_np[b:b + len(keep)], np.array(keep, np.int32)), i
    # K/V of sampled moved rows (every layer and kv head), read before the
    # compaction from the slots that hold their positions
    moved = [(i, s_) for i, keep in sel_o.items() for s_, pos in enumerate(keep) if pos != s_]
    assert moved, "the event moves rows"
    pick = [moved[j] for j in rng.choice(len(moved), size=min(256, len(moved)), replace=False)]
    po0 = meta0["page_off"]
    src_pages = torch.tensor([int(meta0["page_table"][po0[i] + sel_o[i][s_] // P])
                              for i, s_ in pick], device="cuda")
    src_r = torch.tensor([sel_o[i][s_] % P for i, s_ in pick], device="cuda")
    want = [pool[:, src_pages, :, src_r, :].clone() for pool in (kv.k, kv.v)]
    check_rc(L.arbor_compact(kv, k, sel, stt, ws))
    torch.cuda.synchronize()
    assert int(stt) == L.OK
    new_o = O.compact(meta0, ko, sel_o)
    meta1 = _meta(kv)
    for key in ("n_kept", "page_table", "slot_pos"):
        assert np.array_equal(meta1[key], new_o[key]), key
    top = int(meta1["free_top"])
    assert top == int(new_o["free_top"])
    assert np.array_equal(meta1["free_stack"][:top], new_o["free_stack"][:top])
    dst_pages = torch.tensor([int(meta1["page_table"][po0[i] + s_ // P]) for i, s_ in pick],
                             device="cuda")
    dst_r = torch.tensor([s_ % P for _, s_ in pick], device="cuda")
    for pool, w in zip((kv.k, kv.v), want):
        got = pool[:, dst_pages, :, dst_r, :]
        assert torch.equal(got.view(torch.int16), w.view(torch.int16))
    # decode over all 80 layers; sampled outputs against fp64
    Hq = kv.kv_heads * kv.q_per_kv
    nl = active.numel()
    q = st["q_dec"].cuda().contiguous()
    out = torch.empty((nl, kv.layers, Hq, kv.head_dim), device="cuda")
    check_rc(L.arbor_tree_decode_attn(kv, active, 0, kv.layers, q, out, None, 0.0, stt, ws))
    torch.cuda.synchronize()
    assert int(stt) == L.OK
    out_np = out.cpu().numpy()
    po_ = meta1["page_off"]
    scale = 1.0 / math.sqrt(kv.head_dim)
    for b, layer, h in zip(rng.integers(0, nl, 24), rng.integers(0, kv.layers, 24),
                           rng.integers(0, Hq, 24)):
        leaf = int(st["active"][b])
        slots = [(int(meta1["page_table"][po_[x] + s_ // P]), s_ % P)
                 for x in O.chain(parent, leaf) for s_ in range(int(meta1["n_kept"][x]))]
        pg = torch.tensor([x for x, _ in slots], device="cuda")
        rr = torch.tensor([r for _, r in slots], device="cuda")
        g = int(h) // kv.q_per_kv
        K = kv.k[int(layer)][pg, g, rr, :].double().cpu().numpy()
        Vv = kv.v[int(layer)][pg, g, rr, :].double().cpu().numpy()
        qv = q[b, int(layer), int(h)].double().cpu().numpy()
        z = scale * (K @ qv)
        w = np.exp(z - z.max())
        err = np.abs(out_np[b, layer, h] - (w / w.sum()) @ Vv).max()
        assert err <= 2e-3, (b, layer, h, err)
    # every (leaf, query head) of the last layer against the oracle's decode
    _decode_layers_vs_oracle(kv, st, out_np, q, [kv.layers - 1])


def test_dpts_wide_frontier():
    """DPTS-like frontier: 341 nodes of 128 tokens, 16 active leaves decoding."""
    cfg = synth.CONFIGS["dpts"]
    st = synth.build_config(cfg, device="cuda")
    kv = L.kv_state_from(st, "cuda")
    p = st["params"]
    V, N, P = kv.num_nodes, kv.num_tokens, kv.page_size
    parent = st["parent"].tolist()
    ws = _workspace(kv, st, V)
    # score on a sample of observers, against the oracle on the slice layers
    sample = [0, 3, 21, V - 1, V - 64, V - 128]
    idx = [st["observers"].tolist().index(j) for j in sample]
    q_s = st["q_win"][idx].contiguous()
    A, rows, a, s = _gpu_score(kv, st, torch.tensor(sample, dtype=torch.int32, device="cuda"),
                               q_s.cuda(), p, ws)
    Ao, ro, ao, so = _oracle_score(kv, st, sample, np_float(q_s), p)
    _close(A.cpu().numpy(), Ao)
    assert np.array_equal(rows.cpu().numpy(), ro)
    _close(s.cpu().numpy(), so)
    # one eviction event for the 16 leaves with a synthetic score and attention
    rng = np.random.default_rng(2)
    s_full = torch.tensor(rng.random(V).astype(np.float32), device="cuda")
    A_full = torch.tensor((np.round(rng.random(N) * 16) / 16).astype(np.float32), device="cuda")
    active = st["active"].cuda()
    k = torch.empty(V, dtype=torch.int32, device="cuda")
    delta = torch.empty_like(k)
    on_path = torch.empty(V, dtype=torch.uint8, device="cuda")
    stt = status()
    check_rc(L.arbor_allocate(kv, active, st["budget"], s_full, p, k, delta, on_path, stt, ws))
    sel = torch.full((N,), -7, dtype=torch.int32, device="cuda")
    check_rc(L.arbor_select(kv, A_full, k, p, sel, stt))
    check_rc(L.arbor_compact(kv, k, sel, stt, ws))
    torch.cuda.synchronize()
    assert int(stt) == L.OK
    meta0 = _meta(L.kv_state_from(st, "cuda"))            # the generator's (pristine) metadata
    ko, _, _, so_ = O.allocate(meta0["parent"], meta0["n_full"], meta0["n_kept"],
                               st["active"].tolist(), st["budget"], s_full.cpu().numpy(), p)
    assert np.array_equal(k.cpu().numpy(), ko) and so_ == O.OK
    sel_o, _ = O.select(meta0, A_full.cpu().numpy(), ko, p["l_tail"], p["select_mode"])
    sel_np = sel.cpu().numpy()
    for i, keep in sel_o.items():
        b = int(meta0["tok_off"][i])
        assert np.array_equal(sel_np[b:b + len(keep)], np.array(keep, np.int32)), i
    new_o = O.compact(meta0, ko, sel_o)
    meta1 = _meta(kv)
    for key in ("n_kept", "page_table", "slot_pos"):
        assert np.array_equal(meta1[key], new_o[key]), key
    # resident rows of sampled compacted blocks equal the host store rows
    po_ = meta1["page_off"]
    for i in rng.choice(sorted(sel_o), size=8, replace=False):
        c = int(meta1["n_kept"][i])
        pg = torch.tensor([int(meta1["page_table"][po_[i] + s_ // P]) for s_ in range(c)],
                          device="cuda")
        rr = torch.tensor([s_ % P for s_ in range(c)], device="cuda")
        pos = torch.tensor(sel_o[int(i)])
        base = int(meta1["tok_off"][i])
        for pool, store in ((kv.k, st["host_k"]), (kv.v, st["host_v"])):
            got = pool[:, pg, :, rr, :].cpu()
            assert torch.equal(got.view(torch.int16), store[base + pos].view(torch.int16)), i
    # decode of the 16 leaves over all layers; sampled outputs against fp64
    Hq = kv.kv_heads * kv.q_per_kv
    nl = active.numel()
    q = st["q_dec"].cuda().contiguous()
    out = torch.empty((nl, kv.layers, Hq, kv.head_dim), device="cuda")
    check_rc(L.arbor_tree_decode_attn(kv, active, 0, kv.layers, q, out, None, 0.0, stt, ws))
    torch.cuda.synchronize()
    assert int(stt) == L.OK
    out_np = out.cpu().numpy()
    scale = 1.0 / math.sqrt(kv.head_dim)
    for b, layer, h in zip(rng.integers(0, nl, 48), rng.integers(0, kv.layers, 48),
                           rng.integers(0, Hq, 48)):
        leaf = int(st["active"][b])
        slots = [(int(meta1["page_table"][po_[x] + s_ // P]), s_ % P)
                 for x in O.chain(parent, leaf) for s_ in range(int(meta1["n_kept"][x]))]
        pg = torch.tensor([x for x, _ in slots], device="cuda")
        rr = torch.tensor([r for _, r in slots], device="cuda")
        g = int(h) // kv.q_per_kv
        K = kv.k[int(layer)][pg, g, rr, :].double().cpu().numpy()
        Vv = kv.v[int(layer)][pg, g, rr, :].double().cpu().numpy()
        qv = q[b, int(layer), int(h)].double().cpu().numpy()
        z = scale * (K @ qv)
        w = np.exp(z - z.max())
        err = np.abs(out_np[b, layer, h] - (w / w.sum()) @ Vv).max()
        assert err <= 2e-3, (b, layer, h, err)
    # the same decode with the decode-time credit on the slice layers: bitwise
    # the same outputs, and A / rows_seen against the oracle on those layers
    # (16 leaves: more than 16 query rows per kv head on the shared ancestors)
    sl = st["slice_layers"]
    A0 = torch.zeros(N, device="cuda")
    r0 = torch.zeros(V, dtype=torch.int64, device="cuda")
    out2 = torch.empty_like(out)
    check_rc(L.arbor_tree_decode_attn_scored(kv, active, 0, kv.layers, q, out2, None, 0.0, sl, 0,
                                             A0, r0, stt, ws))
    torch.cuda.synchronize()
    assert int(stt) == L.OK
    assert torch.equal(out2.view(torch.int32), out.view(torch.int32))
    ost_sl = _meta(kv, k=kv.k[sl].float().cpu().numpy())
    Ao, ro = O.decode_credit(ost_sl, st["active"].tolist(), 0, np_float(q[:, sl]), kv.q_per_kv,
                             list(range(len(sl))), np.zeros(N, np.float32), np.zeros(V, np.int64))
    _close(A0.cpu().numpy(), Ao)
    assert np.array_equal(r0.cpu().numpy(), ro)
