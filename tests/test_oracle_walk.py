"""Pins of the oracle's event-driven controller (Alg. 2) over a walk:

* after every Transition the whole Path* of the new leaf is resident (full
  protection with lazy rehydration, invariant (i)), and every resident row's
  K/V equals the token-span record of its position (eviction is extractive,
  rehydration restores the full-retention bytes);
* the budget holds after every event that reports OK, and after a Pressure
  event the resident tokens are within B - delta;
* token conservation: resident tokens after the walk = before + restored -
  evicted, summed over the per-event statistics, and each row's resident
  count equals the pool's count after that event;
* no page is lost or duplicated;
* a budget of every token evicts and restores nothing.
"""
import math

import numpy as np
import pytest

from oracle import arbor_oracle as O
from paper_2605_22106_amd import synth
from tests.helpers import np_float, oracle_state

BASE = dict(alpha_max=math.inf, gamma=2.0, lambda_d=0.0, lambda_delta=0.5, eta=0.8, r_min=0.05,
            k_min=2, l_tail=4, theta=(1.0, 1.0, 1.0), select_mode=0, score_self_window=0)


def _tree(seed, scored=False):
    parent, n_full = synth.complete_tree(3, 3, 48, 20)
    st = synth.build_state(parent, n_full, layers=2, kv_heads=1, q_per_kv=2, head_dim=64,
                           dtype="f32", seed=seed, shuffle_pages=True, spare_pages=6,
                           window=4, slice_layers=[0, 1], active=[13])
    targets = synth.walk_targets(parent, 30, 0.3, seed, 13)
    q = None
    if scored:
        import torch
        g = torch.Generator().manual_seed(seed)
        q = torch.randn((len(targets), 2, 2, 4, 64), generator=g).numpy()
    return st, parent, n_full, targets, q


def _resident_rows_match_record(st, host_k, host_v):
    P = st["page_size"]
    for i in range(len(st["parent"])):
        base = int(st["tok_off"][i])
        for (_, page, r, pos) in O.retained(st, i):
            assert np.array_equal(st["k"][:, page, :, r, :], host_k[base + pos]), (i, pos)
            assert np.array_equal(st["v"][:, page, :, r, :], host_v[base + pos]), (i, pos)
    used = sum(-(-int(c) // P) for c in st["n_kept"])
    top = int(st["free_top"])
    assert used + top == st["k"].shape[1]
    pages = [int(st["page_table"][int(st["page_off"][i]) + q])
             for i in range(len(st["parent"])) for q in range(-(-int(st["n_kept"][i]) // P))]
    pages += [int(x) for x in st["free_stack"][:top]]
    assert sorted(pages) == list(range(st["k"].shape[1]))


@pytest.mark.parametrize("seed,margin,scored", [(0, 0, False), (1, 12, False), (2, 0, True),
                                                (3, 20, True)])
def test_walk_invariants(seed, margin, scored):
    st0, parent, n_full, targets, q = _tree(seed, scored)
    ost = oracle_state(st0)
    hk, hv = np_float(st0["host_k"]), np_float(st0["host_v"])
    N = int(st0["num_tokens"])
    budget = int(0.3 * N)
    rng = np.random.default_rng(seed)
    s = rng.random(len(parent)).astype(np.float32)
    A = rng.random(N).astype(np.float32)
    rows = np.zeros(len(parent), np.int64)
    before = int(np.sum(ost["n_kept"]))
    # event by event, so that the state after each one can be inspected
    st, total_restored, total_evicted = ost, 0, 0
    for e, leaf in enumerate(targets):
        st, A, rows, s, stats, status = O.walk(
            st, [leaf], budget, s, A, rows, BASE, hk, hv, pressure_margin=margin,
            q_win=None if q is None else q[e:e + 1], window=4, slice_layers=[0, 1], q_per_kv=2,
            v_sig=np_float(st0["v_sig"]), u_sig=np_float(st0["u_sig"]))
        assert status >= 0
        row = stats[0]
        resident = int(np.sum(st["n_kept"]))
        assert row[0] == resident
        total_restored += int(row[1])
        total_evicted += int(row[2])
        for a in O.chain(parent, leaf):                       # invariant (i)
            assert int(st["n_kept"][a]) == n_full[a]
        if status == O.OK:
            assert resident <= budget
            if row[3]:
                assert resident <= budget - margin
        _resident_rows_match_record(st, hk, hv)
    assert int(np.sum(st["n_kept"])) == before + total_restored - total_evicted
    assert total_restored > 0 and total_evicted > 0


def test_walk_in_one_call_equals_event_by_event():
    st0, parent, n_full, targets, q = _tree(5, scored=True)
    ost = oracle_state(st0)
    hk, hv = np_float(st0["host_k"]), np_float(st0["host_v"])
    N = int(st0["num_tokens"])
    s = np.full(len(parent), 0.5, np.float32)
    A = np.zeros(N, np.float32)
    rows = np.zeros(len(parent), np.int64)
    kw = dict(pressure_margin=10, window=4, slice_layers=[0, 1], q_per_kv=2,
              v_sig=np_float(st0["v_sig"]), u_sig=np_float(st0["u_sig"]))
    one = O.walk(ost, targets, int(0.3 * N), s, A, rows, BASE, hk, hv, q_win=q, **kw)
    st, a_, r_, s_ = ost, A, rows, s
    rows_stats = []
    for e, leaf in enumerate(targets):
        st, a_, r_, s_, stt, status = O.walk(st, [leaf], int(0.3 * N), s_, a_, r_, BASE, hk, hv,
                                            q_win=q[e:e + 1], **kw)
        rows_stats.append(stt[0])
    assert np.array_equal(one[4], np.array(rows_stats))
    assert np.array_equal(one[1], a_) and np.array_equal(one[3], s_)
    for key in ("n_kept", "page_table", "slot_pos"):
        assert np.array_equal(one[0][key], st[key])


def test_full_budget_walk_changes_nothing():
    st0, parent, n_full, targets, _ = _tree(7)
    ost = oracle_state(st0)
    hk, hv = np_float(st0["host_k"]), np_float(st0["host_v"])
    N = int(st0["num_tokens"])
    st, _, _, _, stats, status = O.walk(ost, targets, N, np.full(len(parent), 0.5, np.float32),
                                        np.zeros(N, np.float32), np.zeros(len(parent), np.int64),
                                        BASE, hk, hv)
    assert status == O.OK
    assert np.all(stats[:, 1:] == 0) and np.all(stats[:, 0] == N)
    for key in ("n_kept", "page_table", "slot_pos"):
        assert np.array_equal(st[key], ost[key])
