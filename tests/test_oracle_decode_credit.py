"""Pins of the oracle's decode-time credit of accumulated attention
(Sec. 4 Execution (iii): A_i(t) summed over later queries u > b_i, a thin
slice of layers and all heads, from weights the decoding step computes).

* a hand-computed three-token example (softmax of known logits);
* identical keys: every query spreads its mass uniformly, closed form;
* a decoding query is the window query at the leaf's newest position, so the
  credit equals the observation-window score with W = 1 (pinned separately
  against a dense causal softmax) for both crediting modes;
* the decode attention's own LSE: the credited mass plus the leaf's own mass
  of one query is 1.
"""
import math

import numpy as np
import pytest

from oracle import arbor_oracle as O
from paper_2605_22106_amd import synth
from tests.helpers import oracle_state


def _state(parent, n_full, L=2, Hkv=2, G=2, d=64, seed=0, identical=False, active=None):
    st = synth.build_state(parent, n_full, layers=L, kv_heads=Hkv, q_per_kv=G, head_dim=d,
                           dtype="f32", seed=seed, page_size=4, shuffle_pages=True,
                           identical_keys=identical, active=active,
                           heavy_frac=0.0 if identical else 0.1)
    return st, oracle_state(st)


def test_hand_example():
    """Root with keys e0, e1, a leaf with key 0; q = 2 e0, scale 1/2: logits
    (1, 0, 0), so the root gets e/(e+2) and 1/(e+2); the leaf's own token is
    not credited (and is with self_window only if it is not the newest)."""
    st, ost = _state([-1, 0], [2, 1], L=1, Hkv=1, G=1, d=4, active=[1])
    k = np.zeros_like(ost["k"])
    pt = ost["page_table"]
    k[0, pt[0], 0, 0, :] = [1, 0, 0, 0]
    k[0, pt[0], 0, 1, :] = [0, 1, 0, 0]
    ost["k"] = k
    q = np.zeros((1, 1, 1, 4))
    q[0, 0, 0, 0] = 2.0
    A0 = np.array([0.25, 0.0, 7.0], np.float32)
    A, rows = O.decode_credit(ost, [1], 0, q, 1, [0], A0, np.zeros(2, np.int64))
    e = math.e
    assert np.allclose(A, [0.25 + e / (e + 2), 1 / (e + 2), 7.0], rtol=0, atol=1e-7)
    assert rows.tolist() == [1, 0]
    A1, rows1 = O.decode_credit(ost, [1], 0, q, 1, [0], A0, np.zeros(2, np.int64), self_window=1)
    assert np.array_equal(A1, A)               # the leaf's one token is its newest
    assert rows1.tolist() == [1, 1]


def test_identical_keys_uniform_closed_form():
    parent, n_full = synth.complete_tree(2, 2, 9, 5)
    leaves = [3, 5, 6]
    st, ost = _state(parent, n_full, identical=True, active=leaves, seed=2)
    rng = np.random.default_rng(2)
    n_kept = np.array([int(rng.integers(1, n + 1)) for n in ost["n_full"]])
    keep = {i: sorted(rng.choice(int(ost["n_full"][i]), size=int(n_kept[i]), replace=False))
            for i in range(len(parent))}
    sel = {i: [int(p) for p in keep[i]] for i in keep if n_kept[i] < ost["n_full"][i]}
    ost = O.compact(ost, n_kept, sel)
    q = np.random.default_rng(3).standard_normal((3, 2, 4, 64))
    S = [0, 1]
    A, rows = O.decode_credit(ost, leaves, 0, q, 2, S, np.zeros(int(ost["tok_off"][-1])),
                              np.zeros(len(parent), np.int64))
    want = np.zeros(int(ost["tok_off"][-1]))
    want_rows = np.zeros(len(parent), np.int64)
    for leaf in leaves:
        ch = O.chain(parent, leaf)
        C = sum(int(ost["n_kept"][a]) for a in ch)
        for a in ch[:-1]:
            for p in keep[a]:
                want[int(ost["tok_off"][a]) + p] += len(S) * 4 / C
            want_rows[a] += len(S) * 4
    assert np.allclose(A, want, rtol=1e-6, atol=1e-7)
    assert np.array_equal(rows, want_rows)


@pytest.mark.parametrize("self_window", [0, 1])
@pytest.mark.parametrize("seed", range(3))
def test_equals_window_score_with_one_query(self_window, seed):
    """A decoding query is the window query u = n_l - 1 of an observer l."""
    parent, n_full = synth.random_tree(12, 20, seed, min_tokens=1)
    leaves = [i for i in range(12) if i not in parent][:3]
    st, ost = _state(parent, n_full, L=3, seed=seed, active=leaves)
    rng = np.random.default_rng(seed)
    k = np.array([int(rng.integers(0, c + 1)) for c in ost["n_kept"]])
    sel, _ = O.select(ost, rng.random(int(ost["tok_off"][-1])).astype(np.float32), k, 2)
    ost = O.compact(ost, k, sel)
    l0, S = 1, [1, 2]
    q = rng.standard_normal((len(leaves), 2, 4, 64)).astype(np.float32)
    A0 = rng.random(int(ost["tok_off"][-1])).astype(np.float32)
    r0 = np.arange(12, dtype=np.int64)
    A, rows = O.decode_credit(ost, leaves, l0, q, 2, S, A0, r0, self_window=self_window)
    q_win = np.stack([q[:, l - l0] for l in S], axis=1)[:, :, :, None, :]
    As, rs, _, _ = O.score(ost, leaves, q_win, 1, S, 2, np.zeros(12), np.zeros(12), A0, r0,
                           self_window=self_window)
    assert np.allclose(A, As, rtol=1e-6, atol=0)
    assert np.array_equal(rows, rs)


def test_credit_plus_own_mass_is_one_per_query():
    """One leaf, one slice layer, one head: the weights of the credited tokens
    and of the leaf's own tokens add to 1, the latter from the decode
    attention's LSE (exp(z - lse) summed over the own keys)."""
    parent, n_full = [-1, 0, 1], [11, 7, 5]
    st, ost = _state(parent, n_full, L=1, Hkv=1, G=1, d=64, seed=5, active=[2])
    q = np.random.default_rng(5).standard_normal((1, 1, 1, 64))
    A, _ = O.decode_credit(ost, [2], 0, q, 1, [0], np.zeros(23), np.zeros(3, np.int64))
    _, lse = O.tree_decode_attn(ost, [2], 0, 1, q, 1)
    K = ost["k"][0, :, 0]                                   # [pages][P][d]
    own = [K[p, r] for (_, p, r, _) in O.retained(ost, 2)]
    z_own = np.array(own, np.float64) @ q[0, 0, 0] / 8.0
    own_mass = np.exp(z_own - lse[0, 0, 0]).sum()
    assert abs(A[:18].astype(np.float64).sum() + own_mass - 1.0) < 1e-6
    assert not A[18:].any()
