"""Pins of the QualityDiversitySelect oracle (oracle/qds.py) against what the
seeding passage and arithmetic fix: invariance of the sketch under row
relabelling, the co-assignment counts of a single swap in closed form, row
features of a hand-worked instance, the projection signs against numpy's own
Philox, and the greedy rule on constructed candidate sets."""
import numpy as np
import pytest

import oracle as O
from oracle import qds
import synth


def _prob(D=2, G=1, C=8, k=1, P=2, L=1, E=2, N=4):
    return O.Problem(N, L, E, k, P, D, G, list(np.arange(D) // (D // G)), C, [4096], [1])


def test_features_of_a_hand_worked_row():
    # one layer, two ranks, two slots; row 0 holds samples 0 (t=4) and 1 (t=2)
    # in slots 0 and 1, row 1 holds samples 2 (t=3) and 3 (t=1).
    prob = _prob(D=2, G=1, C=8, k=1, P=2, L=1)
    t = np.array([4, 2, 3, 1])
    q = np.array([[[3, 1]], [[0, 2]], [[1, 2]], [[1, 0]]], dtype=np.int32)
    H = qds.row_features(prob, t, q, 2, np.array([0, 1, 2, 3]))
    one = 1 << qds.QDS_FRAC
    # row 0: T = 6 of D C = 16; Q = 16 + 4 = 20 of D C^2 = 128;
    # W = (3, 1) + (0, 2) = (3, 3), max 3 of k D C = 16
    assert H[0].tolist() == [6 * one // 16, 20 * one // 128, 3 * one // 16]
    # row 1: T = 4, Q = 10, W = (2, 2), max 2
    assert H[1].tolist() == [4 * one // 16, 10 * one // 128, 2 * one // 16]


def test_features_take_the_max_per_shard():
    # two shards of one slot each: the layer profile is max_p over each shard
    # separately, then summed (not the max of the sum)
    prob = _prob(D=2, G=2, C=8, k=1, P=2, L=1)
    t = np.array([4, 4])
    q = np.array([[[4, 0]], [[0, 4]]], dtype=np.int32)
    H = qds.row_features(prob, t, q, 1, np.array([0, 1]))
    one = 1 << qds.QDS_FRAC
    assert H[0, 2] == (4 + 4) * one // 16


def test_projection_signs_follow_numpys_philox():
    F, seed = 67, 2021
    U = qds.directions(F, seed)
    for kk in range(qds.QDS_Q):
        # numpy increments its 256-bit counter before each block: start one below
        c = (kk | (qds.QDS_TAG << 192)) - 1
        prev = np.array([(c >> (64 * w)) & (2**64 - 1) for w in range(4)], dtype=np.uint64)
        gen = np.random.Philox(key=np.array([seed, 0], dtype=np.uint64), counter=prev)
        words = gen.random_raw(4)
        bits = [(int(words[f // 64]) >> (f % 64)) & 1 for f in range(F)]
        assert U[kk].tolist() == [1 if b else -1 for b in bits]


def _small():
    w = synth.make_tiny_random(5, n=40, layers=3, experts=8, top_k=2, ranks=4, dp=4, edp=2, cap=300,
                               tmin=5, tmax=120)
    pd = synth.window_problem(w)
    pb = O.Problem.from_dict(pd)
    slot, _ = O.place(O.aggregate(w.demand), w.n_ranks)
    q = O.project(w.demand, slot, w.n_ranks)
    pr = O.pack_rows(pb, w.lengths, q, 3, 8, 4, 6)
    assert pr["rc"] == 0
    return w, pb, q, pr


def _relabel_rows(x, D, perm):
    return perm[x // D] * D + x % D


def test_sketch_and_coassignment_ignore_row_labels():
    w, pb, q, pr = _small()
    R, D = pr["r_star"], w.n_dp
    x = pr["population"][0]
    perm = np.roll(np.arange(R), 1)
    y = _relabel_rows(x, D, perm)
    U = qds.directions(2 + w.n_layers, 7)
    px = qds.sketch(qds.row_features(pb, w.lengths, q, R, x), U)
    py = qds.sketch(qds.row_features(pb, w.lengths, q, R, y), U)
    assert np.array_equal(px, py)
    assert qds.coassignment(pb, x, y) == (0, 0)
    assert qds.distance_numerator(pb, R, x, y, px, py) == 0


def test_coassignment_of_one_swap_in_closed_form():
    w, pb, q, pr = _small()
    D = w.n_dp
    x = pr["population"][0].astype(np.int64)
    sizes = np.bincount(x, minlength=pr["r_star"] * D)
    for (i, j) in [(0, 1), (2, 17), (5, 33)]:
        if x[i] == x[j]:
            continue
        y = x.copy()
        y[i], y[j] = x[j], x[i]
        A, B = qds.coassignment(pb, x, y)
        assert A == sizes[x[i]] + sizes[x[j]]
        ri, rj = x[i] // D, x[j] // D
        row_size = np.bincount(x // D)
        assert B == (0 if ri == rj else row_size[ri] + row_size[rj])


def test_greedy_prefers_the_diverse_candidate_and_penalises_score():
    w, pb, q, pr = _small()
    R, D = pr["r_star"], w.n_dp
    x0 = pr["population"][0]
    twin = _relabel_rows(x0, D, np.roll(np.arange(R), 1))       # the same plan, rows relabelled
    other = pr["population"][1] if not np.array_equal(pr["population"][1], x0) else pr["population"][2]
    # equal primary scores: the twin (distance 0) comes last
    order = qds.select(pb, w.lengths, q, R, [x0, twin, other], np.array([100, 100, 100]), 9)
    assert order.tolist() == [0, 2, 1]
    # a primary score far above the winner's outweighs any distance (d <= (2 + F) / 3)
    order = qds.select(pb, w.lengths, q, R, [x0, twin, other], np.array([100, 100, 10**6]), 9)
    assert order.tolist() == [0, 1, 2]
    # ties keep the lower index
    order = qds.select(pb, w.lengths, q, R, [x0, twin, twin], np.array([100, 100, 100]), 9)
    assert order.tolist() == [0, 1, 2]


def test_population_repeats_the_selection_order():
    cands = np.arange(12, dtype=np.int32).reshape(3, 4)
    pop = qds.population(cands, np.array([0, 2, 1]), 7)
    assert [int(p[0]) for p in pop] == [0, 8, 4, 0, 8, 4, 0]
