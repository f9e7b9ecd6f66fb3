"""Pins of the oracle's geometry (Sec. 3) and MSVE score (Sec. 4) steps.

Each check is independent of the oracle's own code path: breadth-first search
on the undirected tree, a dense causal softmax over the concatenated token
sequence built from the token-major host store, closed forms (uniform keys,
theta = 0) and the row-mass conservation that any softmax obeys.
"""
import math
from collections import deque

import numpy as np
import pytest
import torch
from scipy.special import softmax, expit

from oracle import arbor_oracle as O
from paper_2605_22106_amd import synth
from tests.helpers import oracle_state, np_float


def bfs_dist(parent, src):
    V = len(parent)
    adj = [[] for _ in range(V)]
    for i in range(1, V):
        adj[i].append(parent[i])
        adj[parent[i]].append(i)
    dist = [-1] * V
    dist[src] = 0
    dq = deque([src])
    while dq:
        x = dq.popleft()
        for y in adj[x]:
            if dist[y] < 0:
                dist[y] = dist[x] + 1
                dq.append(y)
    return dist


@pytest.mark.parametrize("seed", range(6))
def test_geometry_matches_bfs(seed):
    parent, _ = synth.random_tree(40, 5, seed)
    g = torch.Generator().manual_seed(seed)
    active = sorted(set(int(x) for x in torch.randint(0, 40, (3,), generator=g)))
    d, on_path, delta = O.geometry(parent, active)
    root_d = bfs_dist(parent, 0)
    assert list(d) == root_d
    per = [bfs_dist(parent, l) for l in active]
    for i in range(40):
        assert delta[i] == min(p[i] for p in per)
    # Path*: exactly the nodes whose subtree holds an active leaf
    for i in range(40):
        in_sub = any(root_d[l] - root_d[i] == bfs_dist(parent, i)[l] for l in active)
        assert bool(on_path[i]) == in_sub
        if on_path[i] and i > 0:
            assert on_path[parent[i]]          # ancestor-closed
        assert (delta[i] == 0) == (i in active)


def _dense_reference(st, observers, q_win, window, slice_layers, G, scale, self_window, R=None):
    """A via a dense causal softmax over each observer's concatenated chain,
    keys taken from the token-major host store (independent of pages)."""
    parent = st["parent"].tolist()
    n_full = st["n_full"].tolist()
    tok_off = st["tok_off"].tolist()
    hk = np_float(st["host_k"]).astype(np.float64)       # [N][L][Hkv][d]
    N = tok_off[-1]
    A = np.zeros(N)
    Hq = hk.shape[2] * G
    for o, j in enumerate(observers):
        ch = O.chain(parent, j)
        toks, owner, pos = [], [], []
        for a in ch:
            keep = range(n_full[a]) if R is None else R[a]
            for p in keep:
                toks.append(tok_off[a] + p)
                owner.append(a)
                pos.append(p)
        toks, owner, pos = map(np.array, (toks, owner, pos))
        wj = min(window, n_full[j])
        for si, l in enumerate(slice_layers):
            for h in range(Hq):
                Kc = hk[toks, l, h // G, :]
                for t in range(wj):
                    u = n_full[j] - wj + t
                    mask = (owner != j) | (pos <= u)
                    if not mask.any():
                        continue
                    z = scale * (Kc @ q_win[o, si, h, t].astype(np.float64))
                    p = softmax(np.where(mask, z, -np.inf))
                    cred = owner != j
                    if self_window:
                        cred = cred | (pos < u)
                    A[toks[cred & mask]] += p[cred & mask]
    return A


@pytest.mark.parametrize("self_window", [0, 1])
def test_score_matches_dense_causal_softmax(self_window):
    parent, n_full = synth.random_tree(9, 21, 3, min_tokens=3)
    st = synth.build_state(parent, n_full, layers=2, kv_heads=2, q_per_kv=2, head_dim=16,
                           dtype="f32", seed=5, shuffle_pages=True, window=6, page_size=4)
    ost = oracle_state(st)
    q = np_float(st["q_win"])
    obs = st["observers"].tolist()
    scale = 1.0 / math.sqrt(16)
    A, rows, a, s = O.score(ost, obs, q, 6, st["slice_layers"], 2, st["v_sig"].numpy(),
                            st["u_sig"].numpy(), np.zeros(st["num_tokens"], np.float32),
                            np.zeros(9, np.int64), softmax_scale=scale, self_window=self_window)
    ref = _dense_reference(st, obs, q, 6, st["slice_layers"], 2, scale, self_window)
    np.testing.assert_allclose(A, ref, rtol=1e-6, atol=1e-12)


def test_score_with_evictions_matches_dense():
    parent, n_full = synth.random_tree(7, 30, 8, min_tokens=10)
    st = synth.build_state(parent, n_full, layers=1, kv_heads=2, q_per_kv=1, head_dim=8,
                           dtype="f32", seed=2, window=4, page_size=4)
    ost = oracle_state(st)
    # evict by a random selection through the oracle's own compaction
    g = np.random.default_rng(0)
    k = np.array([max(1, c // 3) for c in n_full])
    sel = {i: sorted(g.choice(n_full[i], size=k[i], replace=False).tolist()) for i in range(7)}
    ost2 = O.compact(ost, k, sel)
    q = np_float(st["q_win"])
    scale = 0.5
    A, *_ = O.score(ost2, list(range(7)), q, 4, [0], 1, np.zeros(7), np.zeros(7),
                    np.zeros(st["num_tokens"], np.float32), np.zeros(7, np.int64),
                    softmax_scale=scale)
    ref = _dense_reference(st, list(range(7)), q, 4, [0], 1, scale, 0, R=sel)
    np.testing.assert_allclose(A, ref, rtol=1e-6, atol=1e-12)


def test_score_uniform_keys_closed_form_and_mass():
    """All keys equal: every row spreads 1/|C| over its context."""
    parent, n_full = synth.complete_tree(2, 2, 12, 7)
    st = synth.build_state(parent, n_full, layers=1, kv_heads=1, q_per_kv=2, head_dim=8,
                           dtype="f32", seed=1, window=3, page_size=4, identical_keys=True)
    ost = oracle_state(st)
    q = np_float(st["q_win"])
    V = len(parent)
    A, rows, a, s = O.score(ost, list(range(V)), q, 3, [0], 2, np.zeros(V), np.zeros(V),
                            np.zeros(st["num_tokens"], np.float32), np.zeros(V, np.int64))
    tok_off = st["tok_off"].tolist()
    ref = np.zeros(st["num_tokens"])
    for j in range(V):
        ch = O.chain(parent, j)
        anc_tokens = sum(n_full[a] for a in ch[:-1])
        for t in range(3):
            u = n_full[j] - 3 + t
            C = anc_tokens + u + 1
            for a in ch[:-1]:
                ref[tok_off[a]:tok_off[a + 1]] += 2.0 / C      # two heads
    np.testing.assert_allclose(A, ref, rtol=1e-6)
    # rows_seen: every proper ancestor sees W * Hq rows per descendant observer
    for i in range(V):
        desc = sum(1 for j in range(V) if j != i and i in O.chain(parent, j))
        assert rows[i] == desc * 3 * 2


def test_score_row_mass_bounds():
    """Softmax rows carry unit mass: credited mass per block is in [0, 1] per
    observing row, and crediting the own window only adds mass."""
    parent, n_full = synth.random_tree(8, 18, 11, min_tokens=4)
    st = synth.build_state(parent, n_full, layers=1, kv_heads=2, q_per_kv=1, head_dim=8,
                           dtype="f32", seed=3, window=5, page_size=4)
    ost = oracle_state(st)
    q = np_float(st["q_win"])
    V = len(parent)
    z = np.zeros(st["num_tokens"], np.float32)
    A0, r0, a, s = O.score(ost, list(range(V)), q, 5, [0], 1, np.zeros(V), np.zeros(V), z,
                           np.zeros(V, np.int64))
    A1, r1, _, _ = O.score(ost, list(range(V)), q, 5, [0], 1, np.zeros(V), np.zeros(V), z,
                           np.zeros(V, np.int64), self_window=1)
    rows_total = sum(min(5, n) * 2 for j, n in enumerate(n_full) if j > 0)
    assert np.all(A0 >= 0) and A0.astype(np.float64).sum() <= rows_total + 1e-4
    assert np.all(A1 >= A0)
    for i in range(V):
        if r0[i]:
            assert 0.0 <= a[i] <= 1.0 + 1e-6


def test_msve_closed_form():
    """theta = 0 gives s = sigmoid(0) = 0.5; otherwise s = expit(theta.phi)."""
    parent, n_full = synth.complete_tree(2, 1, 8, 6)
    st = synth.build_state(parent, n_full, layers=1, kv_heads=1, q_per_kv=1, head_dim=4,
                           dtype="f32", seed=0, window=2, page_size=4)
    ost = oracle_state(st)
    q = np_float(st["q_win"])
    v = st["v_sig"].numpy()
    u = st["u_sig"].numpy()
    A, rows, a, s = O.score(ost, [0, 1, 2], q, 2, [0], 1, v, u, np.zeros(20, np.float32),
                            np.zeros(3, np.int64), theta=(0.0, 0.0, 0.0))
    assert np.all(s == np.float32(0.5))
    A, rows, a, s = O.score(ost, [0, 1, 2], q, 2, [0], 1, v, u, np.zeros(20, np.float32),
                            np.zeros(3, np.int64), theta=(0.7, -1.3, 2.0))
    np.testing.assert_allclose(s, expit(0.7 * v - 1.3 * u + 2.0 * a.astype(np.float64)),
                               rtol=1e-6)
    # the root is observed by both children's windows: 2 rows each
    assert rows[0] == 4 and rows[1] == 0
    np.testing.assert_allclose(a[0], A[:8].astype(np.float64).sum() / 4, rtol=1e-6)


def test_heavy_tokens_attract_attention():
    """Statistical sanity: x4-norm keys collect more accumulated attention."""
    cfg = synth.CONFIGS["tiny"]
    st = synth.build_config(cfg)
    ost = oracle_state(st)
    A, *_ = O.score(ost, list(range(7)), np_float(st["q_win"]), cfg.window, cfg.slice_layers,
                    cfg.q_per_kv, st["v_sig"].numpy(), st["u_sig"].numpy(),
                    np.zeros(st["num_tokens"], np.float32), np.zeros(7, np.int64))
    heavy = st["heavy"].numpy()
    root = slice(0, 64)
    assert np.median(A[root][heavy[root]]) > np.median(A[root][~heavy[root]])


def test_uncertainty_eq1():
    assert O.uncertainty(np.zeros(50)) == pytest.approx(0.0, abs=1e-12)
    z = np.full(1000, -60.0)
    z[3] = 0.0
    assert O.uncertainty(z) == pytest.approx(1.0, abs=1e-12)
    # two outcomes with probabilities p, 1-p over a vocabulary of 2
    p = 0.2
    H = -(p * math.log(p) + (1 - p) * math.log(1 - p))
    assert O.uncertainty([math.log(p), math.log(1 - p)]) == pytest.approx(1 - H / math.log(2))
    # top-K with "other": 4 equal logits, K=2 -> outcomes (1/4, 1/4, 1/2)
    H2 = -(2 * 0.25 * math.log(0.25) + 0.5 * math.log(0.5))
    assert O.uncertainty(np.zeros(4), top_k=2) == pytest.approx(1 - H2 / math.log(4))


def test_uncertainty_top_k_against_hand_computed_outcomes():
    # distinct probabilities 0.5, 0.3, 0.15, 0.05 with K = 2: outcomes 0.5, 0.3, other 0.2
    z = [math.log(0.5), math.log(0.3), math.log(0.15), math.log(0.05)]
    H = -(0.5 * math.log(0.5) + 0.3 * math.log(0.3) + 0.2 * math.log(0.2))
    assert O.uncertainty(z, top_k=2) == pytest.approx(1 - H / math.log(4), abs=1e-12)
    # a tie at the K-th value: [e, 1, 1, 1] / S with K = 2 keeps e and one of the 1s
    z = [1.0, 0.0, 0.0, 0.0]
    S = math.e + 3
    p1, p0 = math.e / S, 1 / S
    H = -(p1 * math.log(p1) + p0 * math.log(p0) + 2 * p0 * math.log(2 * p0))
    assert O.uncertainty(z, top_k=2) == pytest.approx(1 - H / math.log(4), abs=1e-12)


def test_uncertainty_top_k_is_a_coarsening():
    # merging outcomes into "other" can only lower the entropy, and K >= |V| is the full sum
    rng = np.random.default_rng(5)
    for _ in range(20):
        z = rng.normal(0, rng.uniform(0.2, 4.0), size=int(rng.integers(2, 300)))
        full = O.uncertainty(z)
        assert 0.0 <= full <= 1.0 + 1e-12
        for k in (1, 3, len(z) - 1):
            assert O.uncertainty(z, top_k=k) >= full - 1e-12
        assert O.uncertainty(z, top_k=len(z)) == pytest.approx(full, abs=1e-12)
