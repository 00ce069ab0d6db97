"""Pins of the cell-count lower bounds (oracle/bounds.py): never above the
exhaustive minimum on small instances, equal to it on constructed ones where
each bound is tight, and equal to the bounds of R_lb on the benchmark
windows (whose FFD row count meets R_lb)."""
import itertools

import numpy as np
import pytest

import oracle as O
from oracle import bounds
import synth


def _min_bins(t, C):
    """Exhaustive minimum number of bins of capacity C (largest item first)."""
    t = sorted(t, reverse=True)
    best = [len(t)]

    def go(i, loads):
        if len(loads) >= best[0]:
            return
        if i == len(t):
            best[0] = len(loads)
            return
        for b in range(len(loads)):
            if loads[b] + t[i] <= C:
                loads[b] += t[i]
                go(i + 1, loads)
                loads[b] -= t[i]
        loads.append(t[i])
        go(i + 1, loads)
        loads.pop()

    go(0, [])
    return best[0]


@pytest.mark.parametrize("seed", range(40))
def test_bound_never_exceeds_the_minimum(seed):
    rng = np.random.default_rng([11, seed])
    C = int(rng.integers(10, 60))
    n = int(rng.integers(1, 9))
    t = rng.integers(1, C + 1, size=n)
    assert bounds.cell_lower_bound(t, C) <= _min_bins(t.tolist(), C)


def test_cardinality_bound_is_tight_for_items_just_above_a_third():
    # nine items of 0.34 C: two per bin at most, so five bins; volume says four
    C = 100
    t = [34] * 9
    assert -(-sum(t) // C) == 4
    assert bounds.cell_lower_bound(t, C) == 5 == _min_bins(t, C)


def test_l2_is_tight_where_volume_and_cardinality_are_not():
    # three 60s and two 45s: no 45 fits beside a 60, so the 45s share a fourth
    # bin.  Volume gives 3, cardinality 3; L2 at alpha = 45 counts the three
    # 60s (J1, above C - 45) and ceil(90 / 100) = 1 more.
    C = 100
    t = [60, 60, 60, 45, 45]
    assert -(-sum(t) // C) == 3
    assert max(-(-sum(1 for v in t if (k + 1) * v > C) // k) for k in range(1, 6)) == 3
    assert bounds.cell_lower_bound(t, C) == 4 == _min_bins(t, C)


def test_rows_round_up_over_the_slots():
    assert bounds.row_lower_bound([34] * 9, 100, 2) == (3, 5)
    assert bounds.row_lower_bound([34] * 9, 100, 1, min_rows=7) == (7, 5)


@pytest.mark.parametrize("name", ["tiny", "small", "mid"])
def test_windows_meet_the_paper_bound(name):
    w = synth.make_window(name)
    t = w.lengths.astype(np.int64)
    C, D = w.capacity, w.n_dp
    r_lb = max(1, -(-int(t.sum()) // (C * D)), -(-int((2 * t > C).sum()) // D))
    r, k = bounds.row_lower_bound(t, C, D)
    pb = O.Problem.from_dict(synth.window_problem(w))
    slot, _ = O.place(O.aggregate(w.demand), w.n_ranks)
    pr = O.pack_rows(pb, w.lengths, O.project(w.demand, slot, w.n_ranks), 1, 2, 1, 2)
    assert r_lb <= r <= pr["r_star"]
    assert pr["certified"] and r == r_lb
