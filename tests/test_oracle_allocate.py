"""Pins of the oracle's tree-aware allocation (Eq. 2, Eq. 3, KKT view, Alg. 2).

* brute force over the global scale alpha: Eq. 2 and Eq. 3 evaluated literally
  (clip, floor, min/max) in exact rational arithmetic at every breakpoint,
  keeping the largest alpha whose total fits the budget;
* Alg. 2's Pressure loop run literally, one token at a time, lowest priority
  first (with the termination fix: nodes at their minimum are skipped);
* the KKT closed form of the relaxed program, solved by a root finder;
* invariants: budget conservation, active-path protection, floors, caps,
  maximality, monotonicity in the budget.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
from scipy.optimize import brentq

from oracle import arbor_oracle as O
from paper_2605_22106_amd import synth

BASE = dict(alpha_max=math.inf, gamma=2.0, lambda_d=0.1, lambda_delta=0.5, eta=0.8,
            r_min=0.05, k_min=2, l_tail=3)


def power(s, gamma):
    """s^gamma: the exact rational power rounded once for integer exponents
    (float(Fraction) rounds to nearest), numpy's power otherwise."""
    if float(gamma).is_integer() and gamma >= 1:
        return float(Fraction(float(s)) ** int(gamma))
    return float(np.power(np.float64(s), gamma))


def weight(s, d, delta, p, on_path=False):
    eta = 1.0 if on_path else p["eta"]
    return float(np.float64(eta) * np.float64(power(s, p["gamma"]))
                 * np.exp(-p["lambda_d"] * d) * np.exp(-p["lambda_delta"] * delta))


def brute_force(parent, n_full, n_kept, active, budget, s, p):
    V = len(parent)
    d, on_path, delta = O.geometry(parent, active)     # geometry is pinned separately
    rehyd = p.get("lazy_rehydration", 1)
    kp = p.get("k_protect", 0)
    # full protection pins Path* blocks (restored to n_i, or kept at c_i without
    # rehydration); floor protection puts them through Eq. 2-3 with eta^0 and
    # a floor of k_protect, up to n_i (c_i without rehydration)
    pinned = n_full if rehyd else n_kept
    free = [i for i in range(V) if not on_path[i] or kp > 0]
    off = [i for i in range(V) if not on_path[i]]
    b_off = budget - sum(pinned[i] for i in range(V) if on_path[i] and kp == 0)
    W = {i: Fraction(weight(s[i], d[i], delta[i], p, bool(on_path[i]))) for i in free}
    rmin = Fraction(p["r_min"])
    cap = {i: (n_full[i] if rehyd else n_kept[i]) if on_path[i] else n_kept[i] for i in free}

    def keep(i, alpha):
        r = min(Fraction(1), max(rmin, alpha * W[i]))
        kk = max(p["k_min"], min(p["l_tail"], n_full[i]), math.floor(r * n_full[i]))
        if on_path[i]:
            kk = max(kk, kp)
        return min(cap[i], min(n_full[i], kk))

    cands = [Fraction(0)]
    for i in free:
        if W[i] > 0:
            cands += [Fraction(j) / (W[i] * n_full[i]) for j in range(1, n_full[i] + 1)]
    if math.isfinite(p["alpha_max"]):
        amax = Fraction(p["alpha_max"])
        cands = [a for a in cands if a <= amax] + [amax]
    best = None
    for a in sorted(set(cands)):
        tot = sum(keep(i, a) for i in free)
        if tot <= b_off:
            best = a
    k = np.zeros(V, dtype=np.int64)
    for i in range(V):
        k[i] = pinned[i] if (on_path[i] and kp == 0) else 0
    if best is not None:
        for i in free:
            k[i] = keep(i, best)
        return k, O.OK
    # Pressure (Alg. 2): floors first, then lower the lowest-priority node by one
    for i in free:
        k[i] = keep(i, Fraction(0))
    prio = {i: weight(s[i], d[i], delta[i], p) for i in off}
    while sum(k[i] for i in free) > b_off:
        movable = [i for i in off if k[i] > min(p["k_min"], n_kept[i])]
        if not movable:
            return k, O.OVER_BUDGET
        j = min(movable, key=lambda i: (prio[i], i))
        k[j] = max(min(p["k_min"], n_kept[j]), k[j] - 1)
    return k, O.OK


def random_case(seed, V=12, max_n=14):
    rng = np.random.default_rng(seed)
    parent, n_full = synth.random_tree(V, max_n, seed, min_tokens=1)
    n_kept = [int(rng.integers(0, n + 1)) if rng.random() < 0.4 else n for n in n_full]
    leaves = [i for i in range(V) if i not in parent]
    active = sorted(rng.choice(leaves, size=min(2, len(leaves)), replace=False).tolist())
    s = rng.random(V).astype(np.float32)
    s[rng.integers(0, V)] = 0.0
    return parent, n_full, n_kept, active, s


@pytest.mark.parametrize("seed", range(40))
def test_allocate_matches_brute_force(seed):
    parent, n_full, n_kept, active, s = random_case(seed)
    p = dict(BASE)
    if seed % 4 == 1:
        p["alpha_max"] = 0.7
    if seed % 4 == 2:
        p.update(gamma=1.0, lambda_d=-0.2)
    if seed % 4 == 3:
        p.update(gamma=3.0)
    total = sum(n_full)
    for rho in (0.2, 0.45, 0.7, 1.0):
        budget = int(rho * total)
        k, delta, on_path, status = O.allocate(parent, n_full, n_kept, active, budget, s, p)
        kb, sb = brute_force(parent, n_full, n_kept, active, budget, s, p)
        assert status == sb
        assert k.tolist() == kb.tolist(), (rho, k, kb)


@pytest.mark.parametrize("seed", range(20))
def test_allocate_invariants(seed):
    parent, n_full, n_kept, active, s = random_case(seed + 100, V=20, max_n=30)
    p = dict(BASE)
    V = len(parent)
    prev = None
    for rho in np.linspace(0.1, 1.0, 10):
        budget = int(rho * sum(n_full))
        k, delta, on_path, status = O.allocate(parent, n_full, n_kept, active, budget, s, p)
        path = [i for i in range(V) if on_path[i]]
        for i in path:
            assert k[i] == n_full[i]                               # invariant (i)
        for i in range(V):
            if not on_path[i]:
                assert k[i] <= n_kept[i]                            # no re-growth off-path
                assert k[i] >= min(p["k_min"], n_kept[i])           # invariant (ii)
        if status == O.OK:
            assert k.sum() <= budget
        floors = {i: O.floor_count(n_full[i], n_kept[i], p) for i in range(V) if not on_path[i]}
        if sum(floors.values()) <= budget - sum(n_full[i] for i in path):
            assert status == O.OK
            for i, f in floors.items():
                assert k[i] >= f                                  # Eq. 3 floors hold
        if prev is not None and status == O.OK:
            assert np.all(k >= prev)                                # monotone in budget
        prev = k if status == O.OK else None


def test_allocate_maximality():
    """No single extra tie group of prices fits: the next breakpoint overflows."""
    parent, n_full = synth.complete_tree(3, 2, 40, 25)
    rng = np.random.default_rng(3)
    s = rng.random(len(parent)).astype(np.float32)
    p = dict(BASE)
    for budget in range(120, 400, 17):          # path 90 + floors 30 and up
        k, _, on_path, st = O.allocate(parent, n_full, n_full, [4], budget, s, p)
        assert st == O.OK and k.sum() <= budget
        kb, _ = brute_force(parent, n_full, n_full, [4], budget, s, p)
        assert k.tolist() == kb.tolist()


def test_kkt_relaxed_solution():
    """K_min = L_tail = r_min = 0 and long blocks: Eq. 2-3 at the budget-meeting
    alpha reproduce the capped KKT allocation k_i = min(n_i, W_i / lambda) of the
    relaxed program with weights W_i = w_i n_i, up to the floor."""
    parent, n_full = synth.complete_tree(4, 2, 3000, 2000)
    rng = np.random.default_rng(7)
    s = (0.2 + 0.8 * rng.random(len(parent))).astype(np.float32)
    p = dict(BASE, k_min=0, l_tail=0, r_min=0.0)
    active = [5]
    d, on_path, delta = O.geometry(parent, active)
    budget = 3000 + 2000 * 2 + 9000
    k, _, _, st = O.allocate(parent, n_full, n_full, active, budget, s, p)
    assert st == O.OK
    off = [i for i in range(len(parent)) if not on_path[i]]
    Wt = np.array([weight(s[i], d[i], delta[i], p) * n_full[i] for i in off])
    n = np.array([n_full[i] for i in off], dtype=np.float64)
    b_off = budget - (3000 + 4000)
    lam = brentq(lambda x: np.minimum(n, Wt / x).sum() - b_off, 1e-9, 1e9)
    kstar = np.minimum(n, Wt / lam)
    got = np.array([k[i] for i in off], dtype=np.float64)
    # the discrete alpha is at least the relaxed one (floor(W/lambda) fits) ...
    assert np.all(got >= np.floor(kstar) - 1e-9)
    assert b_off - len(off) <= got.sum() <= b_off
    # ... and one scalar alpha explains every count: got_i <= alpha W_i < got_i + 1
    assert np.max(got / Wt) < np.min((got + 1) / Wt)


def test_tiny_config_is_over_budget():
    """The tiny configuration's path alone fills a 50 % budget."""
    cfg = synth.CONFIGS["tiny"]
    parent, n_full = synth.complete_tree(2, 2, 64, 32)
    s = np.full(7, 0.5, np.float32)
    k, delta, on_path, st = O.allocate(parent, n_full, n_full, [3], 128, s, cfg.params)
    assert st == O.OVER_BUDGET
    assert on_path.tolist() == [1, 1, 0, 1, 0, 0, 0]
    assert k.tolist() == [64, 32, 2, 32, 2, 2, 2]
    assert delta.tolist() == [2, 1, 3, 0, 2, 4, 4]


@pytest.mark.parametrize("seed", range(20))
def test_allocate_without_rehydration(seed):
    # evicted Path* tokens stay lost (Table 4's ablation): the path keeps c_i and
    # counts c_i, and the tokens it no longer holds go to the off-path blocks
    parent, n_full, n_kept, active, s = random_case(seed + 300)
    p = dict(BASE, lazy_rehydration=0)
    V = len(parent)
    for rho in (0.2, 0.45, 0.7, 1.0):
        budget = int(rho * sum(n_full))
        k, _, on_path, status = O.allocate(parent, n_full, n_kept, active, budget, s, p)
        kb, sb = brute_force(parent, n_full, n_kept, active, budget, s, p)
        assert status == sb and k.tolist() == kb.tolist()
        for i in range(V):
            if on_path[i]:
                assert k[i] == n_kept[i]
        if status == O.OK:
            assert int(np.sum(k)) <= budget
        k1, *_ = O.allocate(parent, n_full, n_kept, active, budget, s, dict(BASE))
        off = [i for i in range(V) if not on_path[i]]
        assert sum(int(k[i]) for i in off) >= sum(int(k1[i]) for i in off)


def test_integer_powers_are_correctly_rounded():
    """s^gamma of Eq. 2 for gamma = 1..4 equals the exact power of the fp32
    score rounded once to fp64."""
    rng = np.random.default_rng(5)
    for x in rng.random(2000).astype(np.float32):
        for g in (1, 2, 3, 4):
            assert O.power(x, float(g)) == float(Fraction(float(x)) ** g)


@pytest.mark.parametrize("seed", range(16))
@pytest.mark.parametrize("gamma", [1.0, 3.0])
def test_negative_zero_score_is_zero(seed, gamma):
    """s = -0 gives w = -0 for an odd gamma; it ranks exactly as s = +0, also in
    the Pressure drain (ties to the lower id), against the brute force."""
    parent, n_full, n_kept, active, s = random_case(seed + 500)
    rng = np.random.default_rng(seed)
    zeros = rng.choice(len(parent), size=4, replace=False)
    s_neg, s_pos = s.copy(), s.copy()
    s_neg[zeros] = np.float32(-0.0)
    s_pos[zeros] = np.float32(0.0)
    p = dict(BASE, gamma=gamma)
    for rho in (0.1, 0.2, 0.45, 1.0):
        budget = int(rho * sum(n_full))
        k, _, _, st = O.allocate(parent, n_full, n_kept, active, budget, s_neg, p)
        k0, _, _, st0 = O.allocate(parent, n_full, n_kept, active, budget, s_pos, p)
        kb, sb = brute_force(parent, n_full, n_kept, active, budget, s_pos, p)
        assert st == st0 == sb
        assert k.tolist() == k0.tolist() == kb.tolist()


def test_scores_outside_the_unit_interval_are_rejected():
    """s_i = clip(sigmoid(.), 0, 1): an off-path score outside [0, 1] is an
    invalid argument, a NaN one is non-finite; Path* scores are never read."""
    parent, n_full = synth.complete_tree(2, 2, 20, 10)
    s = np.full(len(parent), 0.5, np.float32)
    p = dict(BASE)
    for bad, code in ((1.5, O.EINVAL), (-0.25, O.EINVAL), (np.nan, O.ENONFINITE)):
        x = s.copy()
        x[2] = bad                                  # off the path of leaf 3
        assert O.allocate(parent, n_full, n_full, [3], 40, x, p)[3] == code
        x = s.copy()
        x[1] = bad                                  # on the path of leaf 3
        assert O.allocate(parent, n_full, n_full, [3], 40, x, p)[3] in (O.OK, O.OVER_BUDGET)


@pytest.mark.parametrize("seed", range(24))
def test_floor_protection_matches_brute_force(seed):
    """Floor protection (invariant (i) with a floor k_protect): Path* blocks
    take part in Eq. 2-3 without the eta discount, never below k_protect, up
    to n_i (or c_i without rehydration); Pressure drains only off-path
    blocks."""
    parent, n_full, n_kept, active, s = random_case(seed + 700, V=14, max_n=16)
    p = dict(BASE, k_protect=[3, 6, 9, 20][seed % 4], lazy_rehydration=1 - (seed % 5 == 4))
    V = len(parent)
    for rho in (0.15, 0.3, 0.5, 0.75, 1.0):
        budget = int(rho * sum(n_full))
        k, _, on_path, status = O.allocate(parent, n_full, n_kept, active, budget, s, p)
        kb, sb = brute_force(parent, n_full, n_kept, active, budget, s, p)
        assert status == sb, rho
        assert k.tolist() == kb.tolist(), (rho, k, kb)
        for i in range(V):
            if on_path[i]:
                cap = n_full[i] if p["lazy_rehydration"] else n_kept[i]
                assert min(cap, p["k_protect"]) <= k[i] <= cap
        if status == O.OK:
            assert int(np.sum(k)) <= budget


def test_floor_protection_discounts_only_off_path_blocks():
    """Two leaves of equal size and score, one on Path*: with eta < 1 the
    on-path one keeps at least as many tokens; with eta = 1 the same."""
    parent, n_full = [-1, 0, 0], [10, 40, 40]
    s = np.array([0.5, 0.7, 0.7], np.float32)
    for eta, strict in ((0.5, True), (1.0, False)):
        p = dict(BASE, eta=eta, k_protect=1, lambda_delta=0.0, lambda_d=0.0, k_min=0, l_tail=0,
                 r_min=0.0)
        k, _, on_path, st = O.allocate(parent, n_full, n_full, [1], 50, s, p)
        assert st == O.OK and on_path.tolist() == [1, 1, 0]
        assert (k[1] > k[2]) if strict else (abs(int(k[1]) - int(k[2])) <= 1)
