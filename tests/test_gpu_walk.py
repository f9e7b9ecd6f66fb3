"""The deep backtracking tree at full size: 9,841 nodes of 64 tokens (630,784
tokens, 32 layers, 8 KV heads, bf16; 82.7 GB of pool), budget 20 %, and a
random walk with 30 % backtracking.  Every step is one Transition event (Alg. 2):
allocate for the new active node, select + compact the blocks whose count
drops, lazily rehydrate the Path* blocks from the token store.  At this size
the 82.7 GB store is kept in device memory (the entry point takes pinned host
or device memory); the pinned-host path is exercised at the llama8b and dpts
sizes.

Checked at every step: keep-counts bit-exact against the oracle; selections,
page tables, slot maps, resident counts and the free stack bit-exact against
the oracle run on the metadata; all pages accounted for; every Path* block
fully resident afterwards; and, for sampled blocks, every resident row equal
bitwise to the host store row of its position (K and V, all layers and heads).
"""
import numpy as np
import pytest
import torch

from oracle import arbor_oracle as O
from paper_2605_22106_amd import _lib as L
from paper_2605_22106_amd import synth
from tests.gpu_helpers import check_rc, status

pytestmark = pytest.mark.gpu

STEPS = 24


def _meta(kv):
    d = {key: getattr(kv, key).cpu().numpy().astype(np.int64) for key in
         ("parent", "n_full", "tok_off", "page_off", "n_kept", "page_table", "slot_pos",
          "free_stack")}
    d["free_top"] = np.int64(int(kv.free_top.reshape(-1)[0]))
    d["page_size"] = kv.page_size
    npages = kv.slot_pos.shape[0]
    d["k"] = np.zeros((1, npages, 1, kv.page_size, 1), np.float32)   # bytes checked on the GPU
    d["v"] = np.zeros_like(d["k"])
    return d


def _same_meta(a, b):
    for key in ("n_kept", "page_table", "slot_pos"):
        assert np.array_equal(a[key], b[key]), key
    top = int(a["free_top"])
    assert top == int(b["free_top"])
    assert np.array_equal(a["free_stack"][:top], b["free_stack"][:top])


def _rows_match_store(kv, st, meta, i):
    """Resident rows of block i equal the host store rows of their positions."""
    P = kv.page_size
    c = int(meta["n_kept"][i])
    if c == 0:
        return
    po = int(meta["page_off"][i])
    slots = range(c)
    pg = torch.tensor([int(meta["page_table"][po + s // P]) for s in slots], device="cuda")
    rr = torch.tensor([s % P for s in slots], device="cuda")
    pos = torch.tensor([int(meta["slot_pos"][int(meta["page_table"][po + s // P]), s % P])
                        for s in slots])
    base = int(meta["tok_off"][i])
    for pool, store in ((kv.k, st["host_k"]), (kv.v, st["host_v"])):
        got = pool[:, pg, :, rr, :].cpu()                     # [c, L, Hkv, d]
        want = store[(base + pos).to(store.device)].cpu()     # [c, L, Hkv, d]
        assert torch.equal(got.view(torch.int16), want.view(torch.int16)), i


@pytest.fixture(scope="module")
def deep():
    cfg = synth.CONFIGS["deep"]
    st = synth.build_config(cfg, device="cuda", decode_queries=False, host_store="device")
    kv = L.kv_state_from(st, "cuda")
    del st["k"], st["v"]                                      # the pool lives in kv
    return cfg, st, kv


def test_deep_tree_walk_with_lazy_rehydration(deep):
    cfg, st, kv = deep
    p = st["params"]
    V, N, P = kv.num_nodes, kv.num_tokens, kv.page_size
    parent = st["parent"].tolist()
    rng = np.random.default_rng(cfg.seed)
    s = torch.tensor(rng.random(V).astype(np.float32), device="cuda")
    A = torch.tensor(rng.random(N).astype(np.float32), device="cuda")
    s_np, A_np = s.cpu().numpy(), A.cpu().numpy()
    ws = torch.empty(L.arbor_workspace_size(kv, max_context=1024 + 8 * 64), dtype=torch.uint8,
                     device="cuda")
    k = torch.empty(V, dtype=torch.int32, device="cuda")
    delta = torch.empty_like(k)
    on_path = torch.empty(V, dtype=torch.uint8, device="cuda")
    sel = torch.empty(N, dtype=torch.int32, device="cuda")
    host_dummy = np.zeros((N, 1, 1, 1), np.float32)
    targets = synth.walk_targets(parent, STEPS, cfg.walk_backtrack, cfg.seed,
                                 int(st["active"][0]))
    n_rehydrated = 0
    for step, leaf in enumerate(targets):
        print(f"walk step {step}: active node {leaf}", flush=True)
        meta0 = _meta(kv)
        stt = status()
        act = torch.tensor([leaf], dtype=torch.int32, device="cuda")
        check_rc(L.arbor_allocate(kv, act, st["budget"], s, p, k, delta, on_path, stt, ws))
        torch.cuda.synchronize()
        ko, _, po, so = O.allocate(meta0["parent"], meta0["n_full"], meta0["n_kept"], [leaf],
                                   st["budget"], s_np, p)
        assert int(stt) == so, step
        assert np.array_equal(k.cpu().numpy(), ko), step
        sel.fill_(-1)
        check_rc(L.arbor_select(kv, A, k, p, sel, stt))
        check_rc(L.arbor_compact(kv, k, sel, stt, ws))
        torch.cuda.synchronize()
        assert int(stt) in (L.OK, L.OVER_BUDGET), step
        sel_o, _ = O.select(meta0, A_np, ko, p["l_tail"], p["select_mode"])
        sel_np = sel.cpu().numpy()
        for i, keep in sel_o.items():
            b = int(meta0["tok_off"][i])
            assert np.array_equal(sel_np[b:b + len(keep)], np.array(keep, np.int32)), (step, i)
        mid_o = O.compact(meta0, ko, sel_o)
        meta1 = _meta(kv)
        _same_meta(meta1, mid_o)
        check_rc(L.arbor_rehydrate(kv, on_path, st["host_k"], st["host_v"], stt, ws))
        torch.cuda.synchronize()
        assert int(stt) in (L.OK, L.OVER_BUDGET), step
        new_o, rs = O.rehydrate(mid_o, po, host_dummy, host_dummy)
        assert rs == O.OK, step
        meta2 = _meta(kv)
        _same_meta(meta2, new_o)
        used = sum(-(-int(c) // P) for c in meta2["n_kept"])
        assert used + int(meta2["free_top"]) == kv.slot_pos.shape[0], step
        path = O.chain(parent, leaf)
        for i in path:
            assert int(meta2["n_kept"][i]) == int(meta2["n_full"][i]), (step, i)
        back = [i for i in path if int(meta1["n_kept"][i]) < int(meta1["n_full"][i])]
        n_rehydrated += len(back)
        # bytes: the rehydrated blocks and a few compacted ones
        changed = [i for i in sel_o]
        sample = back[:3] + [changed[j] for j in rng.choice(len(changed), size=min(3, len(changed)),
                                                            replace=False)] if changed else back[:3]
        for i in sample:
            _rows_match_store(kv, st, meta2, int(i))
    print(f"walk: {len(targets)} steps, {n_rehydrated} blocks rehydrated", flush=True)
    assert n_rehydrated > 0, "the walk backtracks into evicted blocks"


def test_deep_tree_walk_on_the_device(deep):
    """The full 256-event walk of the deep configuration as one arbor_walk call
    (Alg. 2 on the device: Transition, lazy rehydration, scoring of each new
    leaf's window over its restored chain, eviction, Pressure at B - delta),
    continuing from the state the test above leaves."""
    cfg, st, kv = deep
    p = dict(st["params"])
    V, N, P = kv.num_nodes, kv.num_tokens, kv.page_size
    parent = st["parent"].tolist()
    start = int(st["active"][0])
    targets = synth.walk_targets(parent, cfg.walk_steps, cfg.walk_backtrack, cfg.seed + 1, start)
    steps = len(targets)
    Hq = kv.kv_heads * kv.q_per_kv
    g = torch.Generator(device="cuda").manual_seed(17)
    q = torch.randn((steps, 2, Hq, cfg.window, kv.head_dim), generator=g,
                    device="cuda").to(torch.bfloat16)
    rng = np.random.default_rng(cfg.seed)
    s = torch.tensor(rng.random(V).astype(np.float32), device="cuda")
    A = torch.zeros(N, device="cuda")
    rows = torch.zeros(V, dtype=torch.int64, device="cuda")
    a = torch.empty(V, device="cuda")
    k = torch.empty(V, dtype=torch.int32, device="cuda")
    delta = torch.empty_like(k)
    on_path = torch.empty(V, dtype=torch.uint8, device="cuda")
    sel = torch.empty(N, dtype=torch.int32, device="cuda")
    stats = torch.zeros((steps, 4), dtype=torch.int64, device="cuda")
    ws = torch.empty(L.arbor_workspace_size(kv, max_context=1024 + 8 * 64, max_observers=1,
                                            window=cfg.window, n_slice=2),
                     dtype=torch.uint8, device="cuda")
    margin = 2048
    before = int(kv.n_kept.sum())
    stt = status()
    print(f"device walk: {steps} events", flush=True)
    check_rc(L.arbor_walk(kv, torch.tensor(targets, dtype=torch.int32, device="cuda"),
                          st["budget"], p, A, s, k, delta, on_path, sel, stt, ws,
                          host_k=st["host_k"], host_v=st["host_v"], pressure_margin=margin,
                          q_win=q, window=cfg.window, slice_layers=st["slice_layers"],
                          v_in=st["v_sig"].cuda(), u_in=st["u_sig"].cuda(), rows_seen=rows,
                          a_out=a, stats=stats))
    torch.cuda.synchronize()
    code = int(stt)
    assert code >= 0
    t = stats.cpu().numpy()
    meta = _meta(kv)
    after = int(meta["n_kept"].sum())
    assert t[-1, 0] == after
    assert after == before + int(t[:, 1].sum()) - int(t[:, 2].sum())
    assert t[:, 1].sum() > 0 and t[:, 3].sum() > 0
    if code == L.OK:
        assert np.all(t[:, 0] <= st["budget"])
        assert np.all(t[t[:, 3] == 1, 0] <= st["budget"] - margin)
    used = sum(-(-int(c) // P) for c in meta["n_kept"])
    assert used + int(meta["free_top"]) == kv.slot_pos.shape[0]
    for i in O.chain(parent, targets[-1]):
        assert int(meta["n_kept"][i]) == int(meta["n_full"][i])
    # A grew exactly where the scored leaves' ancestors are
    rows_np = rows.cpu().numpy()
    credited = {a_ for leaf in targets for a_ in O.chain(parent, leaf)[:-1]}
    assert set(np.nonzero(rows_np)[0].tolist()) == credited
    for i in [targets[-1], targets[len(targets) // 2]] + O.chain(parent, targets[0])[:2]:
        _rows_match_store(kv, st, meta, int(i))
