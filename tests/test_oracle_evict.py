"""Pins of the oracle's selection, compaction, rehydration and tree decode
attention (Sec. 4 Execution and lazy rehydration; Alg. 1 Evict; Alg. 2).

* selection against a full lexicographic sort (numpy lexsort) and the
  structural properties of Alg. 1 (extractive, ascending, |R'| = k, tail kept,
  the k <= L_tail branch, nesting across events);
* compaction against the token-major host store: every retained row equals the
  original K/V of its position, byte for byte; pages are conserved;
* rehydrate-after-evict restores the full-retention pool bytes;
* decode attention against torch's scaled-dot-product attention on the CPU in
  float64, and the closed forms of one key and identical keys.
"""
import math

import numpy as np
import pytest
import torch

from oracle import arbor_oracle as O
from paper_2605_22106_amd import synth
from tests.helpers import oracle_state, np_float


def small_state(seed, V=10, max_n=40, P=4, L=2, Hkv=2, d=8, min_n=1):
    parent, n_full = synth.random_tree(V, max_n, seed, min_tokens=min_n)
    st = synth.build_state(parent, n_full, layers=L, kv_heads=Hkv, q_per_kv=1, head_dim=d,
                           dtype="f32", seed=seed, shuffle_pages=True, page_size=P,
                           spare_pages=3)
    return st, oracle_state(st)


def rand_A(st, seed, ties=False):
    rng = np.random.default_rng(seed)
    A = rng.random(st["num_tokens"]).astype(np.float32)
    if ties:
        A = np.round(A * 4).astype(np.float32) / 4          # many exact ties
        A[rng.random(A.shape) < 0.1] = -0.0
    return A


def brute_select(R, A, base, n, k, l_tail, mode):
    R = list(R)
    tail = [p for p in R if p >= n - l_tail]
    if mode == O.TAIL_ONLY or k <= len(tail):
        return R[len(R) - k:] if k else []
    cand = np.array([p for p in R if p < n - l_tail])
    vals = np.array([A[base + p] for p in cand], dtype=np.float64)
    order = np.lexsort((cand, -vals))                         # A desc, then position asc
    return sorted(cand[order[:k - len(tail)]].tolist() + tail)


@pytest.mark.parametrize("seed", range(12))
@pytest.mark.parametrize("mode", [O.TAIL_HEAVY, O.TAIL_ONLY])
def test_select_matches_lexsort(seed, mode):
    st, ost = small_state(seed)
    A = rand_A(st, seed, ties=seed % 2 == 0)
    rng = np.random.default_rng(seed)
    k = [int(rng.integers(0, c + 1)) for c in ost["n_kept"]]
    sel, status = O.select(ost, A, k, 5, mode)
    assert status == O.OK
    for i, c in enumerate(ost["n_kept"]):
        R = [r[3] for r in O.retained(ost, i)]
        if k[i] >= c:
            assert i not in sel
            continue
        want = brute_select(R, A, int(ost["tok_off"][i]), int(ost["n_full"][i]), k[i], 5, mode)
        assert sel[i] == want
        assert set(sel[i]) <= set(R) and sel[i] == sorted(sel[i]) and len(sel[i]) == k[i]
        tail = [p for p in R if p >= ost["n_full"][i] - 5]
        if k[i] >= len(tail):
            assert set(tail) <= set(sel[i])
        else:
            assert sel[i] == R[len(R) - k[i]:]


def test_select_rejects_nan():
    st, ost = small_state(1)
    A = rand_A(st, 1)
    A[3] = np.nan
    k = [0] * len(ost["n_kept"])
    sel, status = O.select(ost, A, k, 2)
    assert status == O.ENONFINITE


def test_negative_zero_ties_positive_zero():
    st, ost = small_state(2, V=1, max_n=12, min_n=12)
    A = np.zeros(12, np.float32)
    A[[1, 5, 7]] = -0.0
    sel, _ = O.select(ost, A, [4], 2)
    assert sel[0] == [0, 1, 10, 11]                        # lowest positions win the tie


def check_pages(ost):
    P = ost["page_size"]
    used = []
    for i in range(len(ost["parent"])):
        po = int(ost["page_off"][i])
        npg = -(-int(ost["n_kept"][i]) // P)
        used += [int(x) for x in ost["page_table"][po:po + npg]]
        cap = int(ost["page_off"][i + 1]) - po
        assert np.all(ost["page_table"][po + npg:po + cap] == -1)
    free = [int(x) for x in ost["free_stack"][:int(ost["free_top"])]]
    allp = sorted(used + free)
    assert allp == list(range(ost["k"].shape[1]))            # no page lost or duplicated
    for pg in free:
        assert np.all(ost["slot_pos"][pg] == -1)


def check_rows_against_store(ost, st):
    hk = np_float(st["host_k"])
    hv = np_float(st["host_v"])
    for i in range(len(ost["parent"])):
        base = int(ost["tok_off"][i])
        prev = -1
        for (s, page, r, pos) in O.retained(ost, i):
            assert pos > prev
            prev = pos
            assert np.array_equal(ost["k"][:, page, :, r, :], hk[base + pos])
            assert np.array_equal(ost["v"][:, page, :, r, :], hv[base + pos])


@pytest.mark.parametrize("seed", range(8))
def test_compact_then_rehydrate_roundtrip(seed):
    st, ost = small_state(seed)
    V = len(ost["parent"])
    rng = np.random.default_rng(seed)
    cur = ost
    # two successive eviction events (nested), then a full rehydration
    for event in range(2):
        A = rand_A(st, seed + event, ties=True)
        k = [int(rng.integers(0, c + 1)) for c in cur["n_kept"]]
        sel, _ = O.select(cur, A, k, 3)
        before = {i: [r[3] for r in O.retained(cur, i)] for i in range(V)}
        cur = O.compact(cur, k, sel)
        for i in range(V):
            after = [r[3] for r in O.retained(cur, i)]
            assert set(after) <= set(before[i])             # extractive, nested
            if i in sel:
                assert after == sel[i]
        check_pages(cur)
        check_rows_against_store(cur, st)
    on_path = np.ones(V, dtype=np.uint8)
    full, status = O.rehydrate(cur, on_path, np_float(st["host_k"]), np_float(st["host_v"]))
    assert status == O.OK
    check_pages(full)
    check_rows_against_store(full, st)
    for i in range(V):
        assert [r[3] for r in O.retained(full, i)] == list(range(int(full["n_full"][i])))


def test_rehydrate_out_of_pages_changes_nothing():
    st, ost = small_state(4)
    V = len(ost["parent"])
    k = [0] * V
    sel, _ = O.select(ost, rand_A(st, 0), k, 3)
    ev = O.compact(ost, k, sel)
    ev["free_top"] = np.int64(2)                         # pretend most pages are taken
    out, status = O.rehydrate(ev, np.ones(V, np.uint8), np_float(st["host_k"]),
                              np_float(st["host_v"]))
    assert status == O.ENOPAGES
    for key in ("n_kept", "page_table", "slot_pos", "free_stack", "k", "v"):
        assert np.array_equal(out[key], ev[key])


def sdpa_chain(st, leaf, l, h, G, scale, R=None):
    """torch's scaled-dot-product attention over the concatenated chain."""
    parent = st["parent"].tolist()
    n_full = st["n_full"].tolist()
    tok_off = st["tok_off"].tolist()
    toks = []
    for a in O.chain(parent, leaf):
        keep = range(n_full[a]) if R is None else R[a]
        toks += [tok_off[a] + p for p in keep]
    K = st["host_k"].to(torch.float64)[toks, l, h // G][None, None]
    Vv = st["host_v"].to(torch.float64)[toks, l, h // G][None, None]
    return K, Vv


@pytest.mark.parametrize("evict", [False, True])
def test_decode_matches_sdpa(evict):
    parent, n_full = synth.random_tree(12, 30, 9, min_tokens=2)
    G = 2
    st = synth.build_state(parent, n_full, layers=3, kv_heads=2, q_per_kv=G, head_dim=16,
                           dtype="f32", seed=9, shuffle_pages=True, page_size=4,
                           active=[7, 11, 3])
    ost = oracle_state(st)
    R = None
    if evict:
        rng = np.random.default_rng(1)
        k = [int(rng.integers(1, c + 1)) for c in ost["n_kept"]]
        sel, _ = O.select(ost, rand_A(st, 5), k, 3)
        ost = O.compact(ost, k, sel)
        R = {i: [r[3] for r in O.retained(ost, i)] for i in range(12)}
    leaves = [7, 11, 3]
    q = np_float(st["q_dec"])[:, 1:3]
    scale = 0.3
    o, lse = O.tree_decode_attn(ost, leaves, 1, 3, q, G, softmax_scale=scale)
    for li, leaf in enumerate(leaves):
        for lr in range(2):
            for h in range(4):
                K, Vv = sdpa_chain(st, leaf, 1 + lr, h, G, scale, R)
                qq = torch.tensor(q[li, lr, h], dtype=torch.float64)[None, None, None]
                ref = torch.nn.functional.scaled_dot_product_attention(qq, K, Vv, scale=scale)
                np.testing.assert_allclose(o[li, lr, h], ref[0, 0, 0].numpy(), rtol=1e-10,
                                           atol=1e-12)
                z = scale * (K[0, 0] @ qq[0, 0, 0])
                assert lse[li, lr, h] == pytest.approx(float(torch.logsumexp(z, 0)), rel=1e-12)


def test_decode_closed_forms():
    # a chain of one single-token node: the output is that token's value
    st = synth.build_state([-1], [1], layers=1, kv_heads=1, q_per_kv=1, head_dim=8, dtype="f32",
                           seed=3, page_size=4, active=[0])
    ost = oracle_state(st)
    o, lse = O.tree_decode_attn(ost, [0], 0, 1, np_float(st["q_dec"]), 1)
    assert np.allclose(o[0, 0, 0], ost["v"][0, 0, 0, 0], rtol=0, atol=1e-15)
    # identical keys: the output is the mean of the values
    parent, n_full = synth.complete_tree(2, 2, 5, 3)
    st = synth.build_state(parent, n_full, layers=1, kv_heads=1, q_per_kv=1, head_dim=8,
                           dtype="f32", seed=4, page_size=4, active=[5], identical_keys=True)
    ost = oracle_state(st)
    o, lse = O.tree_decode_attn(ost, [5], 0, 1, np_float(st["q_dec"]), 1)
    toks = [t for a in O.chain(parent, 5) for t in range(int(st["tok_off"][a]), int(st["tok_off"][a + 1]))]
    mean_v = np_float(st["host_v"])[toks, 0, 0].astype(np.float64).mean(0)
    np.testing.assert_allclose(o[0, 0, 0], mean_v, rtol=1e-12, atol=1e-14)
    z = float(np_float(st["host_k"])[0, 0, 0].astype(np.float64) @ np_float(st["q_dec"])[0, 0, 0]) / math.sqrt(8)
    assert lse[0, 0, 0] == pytest.approx(z + math.log(len(toks)), rel=1e-12)


def _priority_brute_force(R, n, A_of, k, l_tail, mode, n_sinks):
    """The kept set as the first k of one priority list: sinks (lowest position
    first), then -- tail + heavy hitters -- the tail (most recent first) and the
    other tokens by (A desc, position asc), or -- tail-only / sinks + tail --
    the other tokens most recent first."""
    sink = [p for p in R if p < n_sinks]
    rest = [p for p in R if p >= n_sinks]
    if mode == O.TAIL_HEAVY:
        tail = sorted([p for p in rest if p >= n - l_tail], reverse=True)
        head = sorted([p for p in rest if p < n - l_tail], key=lambda p: (-A_of(p) + 0.0, p))
        order = sink + tail + head
    else:
        order = sink + sorted(rest, reverse=True)
    return sorted(order[:k])


@pytest.mark.parametrize("seed", range(30))
@pytest.mark.parametrize("mode", [0, 1, 2])
def test_sinks_and_modes_match_priority_brute_force(seed, mode):
    """Global sinks (the root's first n_sinks positions, Sec. 4 Execution (i))
    and the three intra-block rules of Table 7 against one priority list."""
    rng = np.random.default_rng(seed)
    parent = [-1, 0, 0, 1]
    n_full = [int(x) for x in rng.integers(3, 40, size=4)]
    st = synth.build_state(parent, n_full, layers=1, kv_heads=1, q_per_kv=1, head_dim=64,
                           dtype="f32", seed=seed, active=[3])
    ost = oracle_state(st)
    # a first eviction so that resident sets are ragged (sinks may be gone)
    A0 = rng.random(st["num_tokens"]).astype(np.float32)
    k0 = np.array([int(rng.integers(1, n + 1)) for n in n_full])
    sel0, _ = O.select(ost, A0, k0, 3, O.TAIL_HEAVY, n_sinks=0)
    ost = O.compact(ost, k0, sel0)
    A = (np.round(rng.random(st["num_tokens"]) * 6) / 6).astype(np.float32)
    n_sinks = int(rng.integers(0, 12))
    l_tail = int(rng.integers(0, 6))
    k = np.array([int(rng.integers(0, int(c) + 1)) for c in ost["n_kept"]])
    sel, status = O.select(ost, A, k, l_tail, mode, n_sinks=n_sinks)
    assert status == O.OK
    for i in range(4):
        c = int(ost["n_kept"][i])
        if k[i] >= c:
            assert i not in sel
            continue
        R = [r[3] for r in O.retained(ost, i)]
        base = int(ost["tok_off"][i])
        ns = n_sinks if (i == 0 and mode != O.TAIL_ONLY) else 0
        want = _priority_brute_force(R, n_full[i], lambda p: float(A[base + p]), int(k[i]),
                                     l_tail, mode, ns)
        assert sel[i] == want, (i, mode, n_sinks)
