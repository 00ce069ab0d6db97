"""Pins of the fixed-bin feasibility search (oracle/fixedbin.py): its verdict
equals the exhaustive one (a layout with K non-empty cells exists iff the
minimum bin count is at most K and K is at most N), every solution it
returns is a layout, and the node budget ends the search as unknown."""
import numpy as np
import pytest

from oracle import fixedbin
from test_bound_pins import _min_bins


@pytest.mark.parametrize("seed", range(60))
def test_verdict_matches_exhaustive_search(seed):
    rng = np.random.default_rng([17, seed])
    C = int(rng.integers(10, 60))
    n = int(rng.integers(1, 10))
    t = rng.integers(1, C + 1, size=n)
    mb = _min_bins(t.tolist(), C)
    for K in range(1, n + 2):
        st, nodes, cells = fixedbin.search(t, C, K, 10**6)
        assert st == (fixedbin.FEASIBLE if mb <= K <= n else fixedbin.INFEASIBLE)
        if st == fixedbin.FEASIBLE:
            assert len(cells) == n and cells.min() >= 0 and cells.max() < K
            assert (np.bincount(cells, weights=t, minlength=K) <= C).all()
            assert (np.bincount(cells, minlength=K) >= 1).all()


def test_items_just_above_a_third():
    # nine items of 0.34 C: no four cells hold them, five do
    assert fixedbin.search([34] * 9, 100, 4, 10**6)[0] == fixedbin.INFEASIBLE
    assert fixedbin.search([34] * 9, 100, 5, 10**6)[0] == fixedbin.FEASIBLE


def test_budget_stops_the_search():
    st, nodes, cells = fixedbin.search([34] * 9, 100, 4, 3)
    assert (st, nodes, cells) == (fixedbin.UNKNOWN, 3, None)
