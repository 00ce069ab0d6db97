"""Property-based checks of the oracle (hypothesis): invariants that the
paper's definitions fix for every input, drawn over small random instances.

- LPT (Alg. 1): each layer's placement is a bijection onto the slots with H
  experts per rank, the rank loads are Eq. placement-load of that placement,
  no rank carries more than the H largest expert loads together, and the
  first P experts of the (-L, e) order go to distinct ranks.
- Projection (Eq. physical-rank-demand): the per-sample rank demand keeps the
  logical top-k demand, sum_p q = sum_e a.
- Score (Eqs. 11-15): the fixed-point score equals the exact-rational score,
  and it is a function of the layout's cells, not of their labels inside a
  shard (relabelling the slots of a shard within a row leaves it unchanged).
- Systematic resampling: offspring counts stay within one of P times the
  normalised weight, sum to P, and parents are non-decreasing.
"""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle as O
from oracle import brute

SETTINGS = settings(max_examples=40, deadline=None, suppress_health_check=[HealthCheck.too_slow])


@SETTINGS
@given(st.integers(1, 4), st.integers(1, 4), st.integers(1, 3), st.data())
def test_lpt_bijection_loads_and_bound(P, H, L, data):
    E = P * H
    agg = np.array(data.draw(st.lists(st.lists(st.integers(0, 10**6), min_size=E, max_size=E),
                                      min_size=L, max_size=L)), dtype=np.int64)
    slot, load = O.place(agg, P)
    for l in range(L):
        assert sorted(slot[l].tolist()) == list(range(E))
        assert np.bincount(slot[l] // H, minlength=P).tolist() == [H] * P
        g = np.zeros(P, dtype=np.int64)
        np.add.at(g, slot[l] // H, agg[l])
        assert g.tolist() == load[l].tolist()
        assert int(load[l].max()) <= int(np.sort(agg[l])[::-1][:H].sum())
        # the first P experts in (-L, e) order land on P different ranks
        # (each starts on an empty rank: all ranks are at load 0 or above it)
        first = sorted(range(E), key=lambda e: (-int(agg[l][e]), e))[:P]
        if agg[l][first].min() > 0:
            assert len({int(slot[l][e]) // H for e in first}) == P


@SETTINGS
@given(st.integers(1, 5), st.integers(1, 3), st.integers(1, 3), st.integers(1, 3), st.data())
def test_projection_keeps_the_logical_demand(N, L, P, H, data):
    E = P * H
    demand = np.array(data.draw(st.lists(st.lists(st.lists(st.integers(0, 500), min_size=E, max_size=E),
                                                  min_size=L, max_size=L), min_size=N, max_size=N)),
                      dtype=np.int32)
    perm = np.array([data.draw(st.permutations(list(range(E)))) for _ in range(L)], dtype=np.int32)
    q = O.project(demand, perm, P)
    assert np.array_equal(q.sum(axis=2), demand.sum(axis=2))
    for l in range(L):
        for p in range(P):
            assert np.array_equal(q[:, l, p], demand[:, l, perm[l] // H == p].sum(axis=1))


def _instance(data, D, G):
    R = data.draw(st.integers(1, 3))
    N = data.draw(st.integers(R * D, R * D + 4))
    L = data.draw(st.integers(0, 2))
    P = data.draw(st.sampled_from([1, 2, 3]))
    C = data.draw(st.integers(60, 200))
    t = np.array(data.draw(st.lists(st.integers(1, 20), min_size=N, max_size=N)), dtype=np.int32)
    q = np.array(data.draw(st.lists(st.lists(st.lists(st.integers(0, 15), min_size=P, max_size=P),
                                             min_size=L, max_size=L), min_size=N, max_size=N)),
                 dtype=np.int32).reshape(N, L, P)
    lay = np.array(data.draw(st.permutations(list(range(N))))) % (R * D)
    S = data.draw(st.integers(1, 2))
    alpha = data.draw(st.lists(st.integers(0, 5000), min_size=S, max_size=S))
    beta = data.draw(st.lists(st.integers(0, 3), min_size=S, max_size=S))
    dp = (np.arange(D) // (D // G)).astype(np.int32)
    prob = O.Problem(N, L, P, 1, P, D, G, dp, C, alpha, beta, frac_bits=12)
    return prob, t, q, R, lay.astype(np.int32), dp


@SETTINGS
@given(st.sampled_from([(1, 1), (2, 1), (2, 2), (4, 2)]), st.data())
def test_score_is_exact_and_label_free(DG, data):
    D, G = DG
    prob, t, q, R, lay, dp = _instance(data, D, G)
    st_, s, _, _ = O.score(prob, t, q, R, lay)
    assert st_ == 0
    assert brute.fixed_point_to_fraction(s, prob) == brute.score_exact(prob, t, q, R, lay)
    # relabel the slots of one shard within every row by a permutation
    g = data.draw(st.integers(0, G - 1))
    slots = [d for d in range(D) if dp[d] == g]
    perm = data.draw(st.permutations(slots))
    remap = {a: b for a, b in zip(slots, perm)}
    lay2 = np.array([(c // D) * D + remap.get(c % D, c % D) for c in lay], dtype=np.int32)
    assert O.score(prob, t, q, R, lay2)[1].tolist() == s.tolist()


@SETTINGS
@given(st.integers(2, 64), st.integers(0, 2**32 - 1), st.data())
def test_resample_offspring_and_order(P, V, data):
    E = np.array(data.draw(st.lists(st.floats(0.0, 5e-4), min_size=P, max_size=P))) + 2.0
    par = O.resample_at(E, 1e-4, 7e-5, V)
    assert (np.diff(par) >= 0).all() and par.min() >= 0 and par.max() < P
    counts = np.bincount(par, minlength=P)
    assert counts.sum() == P
    emin = E.min()
    c = 1 / 7e-5 - 1 / 1e-4
    w = np.exp(-(c * ((E - emin) / max(abs(emin), 1.0))))
    share = P * w / w.sum()
    # systematic resampling: floor(P w) or ceil(P w) offspring (up to the
    # quantisation of the weights, which moves a share by far less than 1e-6)
    assert (counts >= np.floor(share - 1e-6)).all() and (counts <= np.ceil(share + 1e-6)).all()
