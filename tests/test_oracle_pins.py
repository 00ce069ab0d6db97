"""Pins of the CPU oracle against what the paper and mathematics fix.

Nothing here compares the oracle with itself: each check uses a library
routine (numpy Philox, numpy sum/einsum, math.exp), exact rationals written
from the paper's normalised equations, hand-traced steps of Alg. 1, the
numbers printed with Fig. 3, or exhaustive search on tiny inputs.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import synth
import oracle as O
from oracle import brute

GOLD = os.path.join(os.path.dirname(__file__), "golden")


# --------------------------------------------------------------------------
# Philox4x64-10 against numpy.random.Philox (numpy increments the counter
# before each block, so block(c) is Philox(counter=c-1).random_raw(4)).
@pytest.mark.parametrize("seed", range(6))
def test_philox_matches_numpy(oracle_mod, seed):
    rng = np.random.default_rng(seed)
    key = rng.integers(0, 2**64, size=2, dtype=np.uint64)
    ctr = rng.integers(0, 2**64, size=4, dtype=np.uint64)
    ctr[0] = max(int(ctr[0]), 1)
    prev = ctr.copy()
    prev[0] -= np.uint64(1)
    ref = np.random.Philox(key=key, counter=prev).random_raw(4)
    got = oracle_mod.philox4x64(ctr, key)
    assert [int(x) for x in got] == [int(x) for x in ref]


def test_philox_counter_carry(oracle_mod):
    # counter (0, 1, 0, 0) is reached from (2^64-1, 0, 0, 0) by numpy's carry.
    key = np.array([2000, 0], dtype=np.uint64)
    prev = np.array([2**64 - 1, 0, 0, 0], dtype=np.uint64)
    ref = np.random.Philox(key=key, counter=prev).random_raw(4)
    got = oracle_mod.philox4x64(np.array([0, 1, 0, 0], dtype=np.uint64), key)
    assert [int(x) for x in got] == [int(x) for x in ref]


# --------------------------------------------------------------------------
# exp_det: error bound against math.exp over [-708, 0].
def _ulp_err(a, b):
    return abs(a - b) / math.ulp(b)


def test_exp_det_error_bound(oracle_mod):
    rng = np.random.default_rng(1)
    xs = np.concatenate([-np.linspace(0.0, 708.0, 20001), -rng.uniform(0, 708, 20000),
                         -rng.uniform(0, 1e-3, 2000), -np.logspace(-300, 2.85, 2000)])
    got = oracle_mod.exp_det(xs)
    worst = max(_ulp_err(g, math.exp(x)) for g, x in zip(got, xs))
    assert worst <= 2.0, worst


def test_exp_det_special_values(oracle_mod):
    assert oracle_mod.exp_det([0.0, -0.0])[0] == 1.0
    assert oracle_mod.exp_det([-0.0])[0] == 1.0
    assert oracle_mod.exp_det([-708.5, -1e9, float("-inf")]).tolist() == [0.0, 0.0, 0.0]
    assert oracle_mod.exp_det([-1e-300])[0] == 1.0


# --------------------------------------------------------------------------
# Aggregation, LPT, projection.
@pytest.mark.parametrize("name", ["tiny", "small"])
def test_aggregate_is_numpy_sum(oracle_mod, name):
    w = synth.make_window(name)
    agg = oracle_mod.aggregate(w.demand)
    assert np.array_equal(agg, w.demand.sum(axis=0, dtype=np.int64))
    # generator invariant: sum_e L[l, e] = k * sum_i t_i for every layer
    assert (agg.sum(axis=1) == w.top_k * int(w.lengths.astype(np.int64).sum())).all()


def test_lpt_hand_traced(oracle_mod):
    # (-L, e) order: e1(9), e2(9), e0(5), e3(1); argmin over (G, p).
    slot, load = oracle_mod.place(np.array([[5, 9, 9, 1]]), 2)
    assert slot.tolist() == [[1, 0, 2, 3]] and load.tolist() == [[14, 10]]
    # a full rank is skipped: rank 1 holds H = 2 experts before e3 arrives.
    slot, load = oracle_mod.place(np.array([[10, 1, 1, 1]]), 2)
    assert slot.tolist() == [[0, 2, 3, 1]] and load.tolist() == [[11, 2]]
    # all-equal loads fill ranks round-robin by index.
    slot, load = oracle_mod.place(np.array([[3, 3, 3, 3, 3, 3]]), 3)
    assert slot.tolist() == [[0, 2, 4, 1, 3, 5]] and load.tolist() == [[6, 6, 6]]


def test_lpt_invariants(oracle_mod):
    w = synth.make_window("small")
    agg = oracle_mod.aggregate(w.demand)
    slot, load = oracle_mod.place(agg, w.n_ranks)
    H = w.n_experts // w.n_ranks
    for l in range(w.n_layers):
        assert sorted(slot[l].tolist()) == list(range(w.n_experts))       # bijection
        assert np.bincount(slot[l] // H, minlength=w.n_ranks).tolist() == [H] * w.n_ranks
        # G_{l,p} (Eq. placement-load) recomputed by numpy
        g = np.zeros(w.n_ranks, dtype=np.int64)
        np.add.at(g, slot[l] // H, agg[l])
        assert np.array_equal(g, load[l])
    assert np.array_equal(load.sum(axis=1), agg.sum(axis=1))


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_projection_is_onehot_einsum(oracle_mod, name):
    w = synth.make_window(name)
    slot, _ = oracle_mod.place(oracle_mod.aggregate(w.demand), w.n_ranks)
    q = oracle_mod.project(w.demand, slot, w.n_ranks)
    H = w.n_experts // w.n_ranks
    onehot = np.zeros((w.n_layers, w.n_experts, w.n_ranks), dtype=np.int64)
    for l in range(w.n_layers):
        onehot[l, np.arange(w.n_experts), slot[l] // H] = 1
    ref = np.einsum("ile,lep->ilp", w.demand.astype(np.int64), onehot)
    assert np.array_equal(q, ref)
    # logical top-k demand is preserved: sum_p q = k t, and q <= min(k, H) t
    t = w.lengths.astype(np.int64)
    assert (q.sum(axis=2) == w.top_k * t[:, None]).all()
    assert (q <= min(w.top_k, H) * t[:, None, None]).all()


def test_fig3_instance(oracle_mod):
    g = json.load(open(os.path.join(GOLD, "fig3_instance.json")))
    demand = np.array(g["demand"], dtype=np.int32)
    agg = oracle_mod.aggregate(demand)
    ident = np.arange(4, dtype=np.int32)[None, :]
    q_id = oracle_mod.project(demand, ident, 2)
    assert q_id.sum(axis=0)[0].tolist() == g["identity_rank_load"]
    for lay in (g["packing_AB_CD"], g["packing_AC_BD"]):
        rows = [q_id[[i for i in range(4) if lay[i] == r]].sum(axis=0)[0] for r in range(2)]
        assert [int(x.max()) for x in rows] == [g["identity_row_peak"]] * 2
    slot, load = oracle_mod.place(agg, 2)
    assert load[0].tolist() == g["lpt_rank_load"]
    q = oracle_mod.project(demand, slot, 2)
    for lay, peaks in ((g["packing_AB_CD"], g["lpt_row_peaks_packing_AB_CD"]),
                       (g["packing_AC_BD"], g["lpt_row_peaks_packing_AC_BD"])):
        rows = [q[[i for i in range(4) if lay[i] == r]].sum(axis=0)[0] for r in range(2)]
        assert [int(x.max()) for x in rows] == peaks
    # Joint score with a = 1, b = 0: U = 4 for {A,B}{C,D}, 3 for {A,C}{B,D}.
    prob = oracle_mod.Problem(4, 1, 4, 1, 2, 1, 1, [0], 8, [4096], [0])
    for lay, u in ((g["packing_AB_CD"], 4), (g["packing_AC_BD"], 3)):
        st, s, _, _ = oracle_mod.score(prob, g["lengths"], q, 2, lay)
        assert st == 0 and brute.fixed_point_to_fraction(s, prob)[0] == u
        # Eq. packing-lower-bound: sum_r max_p W >= max_p L^agg = 8
    st, s, J, _ = oracle_mod.score(oracle_mod.Problem(4, 1, 4, 1, 2, 1, 1, [0], 8, [0], [0]),
                                   g["lengths"], q, 2, g["packing_AC_BD"], want_J=True)
    assert Fraction(int(s[1]), 4096 * 8) * 8 == 8   # meets the bound with equality


# --------------------------------------------------------------------------
# Exact score against exact rationals from the normalised equations.
def _tiny_cases():
    cases = []
    for seed in range(10):
        for (D, G) in ((2, 1), (2, 2), (4, 2), (3, 3)):
            cases.append((seed, D, G))
    return cases


@pytest.mark.parametrize("seed,D,G", _tiny_cases())
def test_score_matches_exact_rationals(oracle_mod, seed, D, G):
    rng = np.random.default_rng([11, seed, D, G])
    n = int(rng.integers(2 * D, 4 * D + 1))
    w = synth.make_tiny_random(seed, n=n, layers=int(rng.integers(0, 4)), experts=4, ranks=2,
                               dp=D, edp=G, cap=40)
    S = int(rng.integers(1, 3))
    alpha = rng.integers(0, 5000, size=S)
    beta = rng.integers(0, 3, size=S)
    prob = oracle_mod.Problem(w.n, w.n_layers, w.n_experts, w.top_k, w.n_ranks, D, G,
                              w.dp_to_edp, 1000, alpha, beta, frac_bits=12)
    slot, _ = oracle_mod.place(oracle_mod.aggregate(w.demand), w.n_ranks)
    q = oracle_mod.project(w.demand, slot, w.n_ranks)
    R = n // D
    for _ in range(8):
        lay = rng.integers(0, R * D, size=n).astype(np.int32)
        lay[: R * D] = rng.permutation(R * D)  # every cell non-empty
        rng.shuffle(lay)
        st, s, J, _ = oracle_mod.score(prob, w.lengths, q, R, lay, want_J=True)
        ref = brute.score_exact(prob, w.lengths, q, R, lay)
        assert st == 0 and ref is not None
        assert brute.fixed_point_to_fraction(s, prob) == ref


def test_score_status_bits(oracle_mod):
    w = synth.make_tiny_random(3, n=6, dp=2, cap=50)
    prob = oracle_mod.Problem.from_dict(synth.window_problem(w))
    q = np.zeros((6, w.n_layers, w.n_ranks), dtype=np.int32)
    t = np.array([10] * 6, dtype=np.int32)
    assert oracle_mod.score(prob, t, q, 2, [0, 1, 2, 3, 0, 1])[0] == 0
    assert oracle_mod.score(prob, t, q, 2, [0, 1, 2, 4, 0, 1])[0] & 1      # id out of range
    assert oracle_mod.score(prob, [50, 1, 1, 1, 1, 1], q, 2, [0, 0, 1, 2, 3, 3])[0] & 2
    st, s, _, _ = oracle_mod.score(prob, t, q, 2, [0, 1, 2, 2, 0, 1])
    assert st & 4 and s.tolist() == [2**63 - 1] * 3                        # empty cell 3


def test_score_special_cases(oracle_mod):
    # L = 0, D = 1, one stage, a = 1, b = 0: s0 = sum t / C for every layout.
    rng = np.random.default_rng(5)
    t = rng.integers(1, 30, size=9).astype(np.int32)
    prob = oracle_mod.Problem(9, 0, 4, 1, 2, 1, 1, [0], 100, [4096], [0])
    q = np.zeros((9, 0, 2), dtype=np.int32)
    for _ in range(5):
        lay = rng.permutation(np.arange(9) % 3).astype(np.int32)
        st, s, _, _ = oracle_mod.score(prob, t, q, 3, lay)
        assert st == 0 and brute.fixed_point_to_fraction(s, prob)[0] == Fraction(int(t.sum()), 100)


@pytest.mark.parametrize("G", [1, 2])
def test_packing_lower_bound_and_invariance(oracle_mod, G):
    # With alpha = beta = 0, J = E, so s1 = 2^F sum_{r,g,l} max_p W, which must
    # be >= 2^F sum_l max_p L^agg_{l,p} (Eq. packing-lower-bound); and the
    # window rank load is packing-invariant (Eq. aggregate-invariance).
    w = synth.make_window("tiny", edp=G)
    slot, load = oracle_mod.place(oracle_mod.aggregate(w.demand), w.n_ranks)
    q = oracle_mod.project(w.demand, slot, w.n_ranks)
    prob = oracle_mod.Problem(w.n, w.n_layers, w.n_experts, w.top_k, w.n_ranks, w.n_dp, G,
                              w.dp_to_edp, w.capacity, [0], [0])
    rng = np.random.default_rng(2)
    bound = int(load.max(axis=1).sum()) << 12
    for _ in range(10):
        lay = rng.permutation(np.arange(w.n) % (9 * w.n_dp)).astype(np.int32)
        st, s, _, _ = oracle_mod.score(prob, np.ones(w.n, dtype=np.int32), q, 9, lay)
        assert st == 0 and s[1] >= bound
        assert np.array_equal(q.sum(axis=0), load)


# --------------------------------------------------------------------------
# Packing: invariants, canonical form by definition, exhaustive minimum R.
@pytest.mark.parametrize("name,G", [("tiny", 1), ("tiny", 2), ("small", 1)])
def test_pack_rows_invariants(oracle_mod, name, G):
    w = synth.make_window(name, edp=G)
    prob = oracle_mod.Problem.from_dict(synth.window_problem(w))
    slot, _ = oracle_mod.place(oracle_mod.aggregate(w.demand), w.n_ranks)
    q = oracle_mod.project(w.demand, slot, w.n_ranks)
    pr = oracle_mod.pack_rows(prob, w.lengths, q, w.seed_pack, 16, 4, w.pop)
    assert pr["rc"] == 0
    R, D, C = pr["r_star"], w.n_dp, w.capacity
    t = w.lengths.astype(np.int64)
    assert R >= pr["r_lb"] >= math.ceil(t.sum() / (C * D))
    assert pr["certified"] == (R == pr["r_lb"])
    nd = min(pr["n_distinct"], w.pop)
    assert 1 <= pr["n_distinct"] <= 16
    pop = pr["population"]
    for m in range(w.pop):
        lay = pop[m]
        st, s, _, _ = oracle_mod.score(prob, w.lengths, q, R, lay)
        assert st == 0 and s.tolist() == pr["scores"][m].tolist()
        assert np.array_equal(pop[m], pop[m % nd])
        if name == "tiny":
            assert np.array_equal(brute.canonical(lay, R, D, w.dp_to_edp), lay)
    keys = [tuple(x) for x in pr["scores"][:nd].tolist()]
    assert keys == sorted(keys)
    distinct = {pop[m].tobytes() for m in range(nd)}
    assert len(distinct) == nd


@pytest.mark.parametrize("seed", range(12))
def test_row_count_vs_exhaustive(oracle_mod, seed):
    rng = np.random.default_rng([3, seed])
    D = int(rng.integers(1, 3))
    n = int(rng.integers(4, 9))
    C = 20
    t = rng.integers(3, C + 1, size=n).astype(np.int32)
    prob = oracle_mod.Problem(n, 1, 2, 1, 2, D, 1, [0] * D, C, [4096], [1])
    q = np.zeros((n, 1, 2), dtype=np.int32)
    q[:, 0, 0] = t
    pr = oracle_mod.pack_rows(prob, t, q, 7, 4, 2, 2)
    rmin = brute.min_rows(t, C, D)
    if rmin is None:
        assert pr["rc"] in (-2, -3)
        return
    assert pr["rc"] == 0
    assert pr["r_star"] >= rmin
    if pr["certified"]:
        assert pr["r_star"] == rmin


def test_ffd_hand_example(oracle_mod):
    # t = 7,6,5,4,3,2 with C = 10, D = 1: R_lb = ceil(27/10) = 3; the three
    # longest open cells [7],[6],[5]; 4 -> cell 1 (6+4), 3 -> cell 0 (7+3),
    # 2 -> cell 2 (5+2).  R* = 3 and the layout is this FFD packing.
    t = np.array([3, 7, 2, 6, 5, 4], dtype=np.int32)
    prob = oracle_mod.Problem(6, 0, 2, 1, 2, 1, 1, [0], 10, [4096], [0])
    q = np.zeros((6, 0, 2), dtype=np.int32)
    pr = oracle_mod.pack_rows(prob, t, q, 1, 2, 1, 1)
    assert pr["rc"] == 0 and pr["r_star"] == 3 and pr["certified"]
    lay = pr["population"][0]
    cells = sorted(sorted(int(t[i]) for i in range(6) if lay[i] == c) for c in range(3))
    assert cells == [[2, 5], [3, 7], [4, 6]]


def test_pack_rows_errors(oracle_mod):
    prob = oracle_mod.Problem(4, 0, 2, 1, 2, 2, 1, [0, 0], 10, [4096], [0])
    q = np.zeros((4, 0, 2), dtype=np.int32)
    assert oracle_mod.pack_rows(prob, [11, 1, 1, 1], q, 1, 2, 1, 1)["rc"] == -2   # t > C
    prob3 = oracle_mod.Problem(3, 0, 2, 1, 2, 2, 1, [0, 0], 10, [4096], [0])
    assert oracle_mod.pack_rows(prob3, [9, 9, 9], np.zeros((3, 0, 2), np.int32), 1, 2, 1, 1)["rc"] == -2
    bad = oracle_mod.Problem(4, 0, 2, 1, 2, 2, 2, [0, 0], 10, [4096], [0])       # shard 1 empty
    assert oracle_mod.pack_rows(bad, [1, 1, 1, 1], q, 1, 2, 1, 1)["rc"] == -1


# --------------------------------------------------------------------------
# Resampling: textbook properties of systematic resampling.
def test_resample_offspring_counts(oracle_mod):
    rng = np.random.default_rng(9)
    for trial in range(30):
        P = int(rng.integers(1, 40))
        e = rng.normal(1.0, 1e-3, size=P)
        t_cur, t_next = 1e-3, 5e-4
        par = oracle_mod.resample(e, t_cur, t_next, seed=trial, level=trial)
        assert np.all(np.diff(par) >= 0) and par.min() >= 0 and par.max() < P
        emin = e.min()
        den = max(abs(emin), 1.0)
        cfac = (1.0 / t_next) - (1.0 / t_cur)
        wq = [int(math.floor(math.ldexp(float(oracle_mod.exp_det([-(cfac * ((x - emin) / den))])[0]), 40)))
              for x in e]
        S = sum(wq)
        cnt = np.bincount(par, minlength=P)
        for j in range(P):
            pw = Fraction(P * wq[j], S)
            assert math.floor(pw) <= cnt[j] <= math.ceil(pw)
        assert cnt.sum() == P


def test_resample_equal_weights_identity(oracle_mod):
    par = oracle_mod.resample(np.full(16, 3.0), 1e-3, 1e-4, seed=4, level=2)
    assert par.tolist() == list(range(16))


# --------------------------------------------------------------------------
# Annealing special cases and exhaustive optimum.
def _tiny_anneal_setup(seed, D=2, G=1, n=8, cap=40, alpha=(4096,), beta=(1,), layers=2):
    w = synth.make_tiny_random(seed, n=n, layers=layers, experts=4, ranks=2, dp=D, edp=G,
                               cap=cap, tmin=2, tmax=cap // 2)
    import oracle as O
    prob = O.Problem(w.n, w.n_layers, w.n_experts, w.top_k, w.n_ranks, D, G, w.dp_to_edp,
                     cap, list(alpha), list(beta))
    slot, _ = O.place(O.aggregate(w.demand), w.n_ranks)
    q = O.project(w.demand, slot, w.n_ranks)
    pr = O.pack_rows(prob, w.lengths, q, seed, 6, 2, 4)
    return w, prob, q, pr


def test_anneal_all_ties_accept_every_feasible(oracle_mod):
    w, prob, q, pr = _tiny_anneal_setup(1, alpha=(0,), beta=(0,), layers=0)
    assert pr["rc"] == 0
    an = oracle_mod.anneal(prob, w.lengths, q, pr["r_star"], pr["population"],
                           synth.anneal_temperatures(5), 64, 3)
    assert an["rc"] == 0
    tr = an["trace"]
    assert (tr[:, :, 6] == tr[:, :, 7]).all() and tr[:, :, 7].sum() > 0


def test_anneal_infinite_temperature_accepts_every_feasible(oracle_mod):
    w, prob, q, pr = _tiny_anneal_setup(2)
    an = oracle_mod.anneal(prob, w.lengths, q, pr["r_star"], pr["population"],
                           [1e300, 1e299, 1e298], 64, 5)
    tr = an["trace"]
    assert an["rc"] == 0 and (tr[:, :, 6] == tr[:, :, 7]).all()


def test_anneal_zero_temperature_is_greedy(oracle_mod):
    # T -> 0: only moves with Delta <= 0 pass; with G = 1 the energy is then
    # non-increasing along every chain, and the trajectory best is terminal.
    w, prob, q, pr = _tiny_anneal_setup(3)
    an = oracle_mod.anneal(prob, w.lengths, q, pr["r_star"], pr["population"],
                           [1e-300], 128, 6, want_steps=True)
    tr = an["trace"][0]
    assert an["rc"] == 0
    assert (tr[:, 0:3] == tr[:, 3:6]).all()
    start = pr["scores"]
    for j in range(len(start)):
        assert tuple(tr[j, 0:3]) <= tuple(start[j])


@pytest.mark.parametrize("seed", range(8))
def test_anneal_never_beats_exhaustive_optimum(oracle_mod, seed):
    w, prob, q, pr = _tiny_anneal_setup(10 + seed, n=7, D=2, cap=36)
    if pr["rc"] != 0:
        pytest.skip("infeasible instance")
    R = pr["r_star"]
    opt = brute.best_score(prob, w.lengths, q, R)
    an = oracle_mod.anneal(prob, w.lengths, q, R, pr["population"],
                           synth.anneal_temperatures(8), 64, seed, check_full=True)
    assert an["rc"] == 0
    got = brute.fixed_point_to_fraction(an["best_score"], prob)
    assert got >= opt
    assert brute.score_exact(prob, w.lengths, q, R, an["best_layout"]) == got


def test_anneal_reaches_optimum_often(oracle_mod):
    hits = tot = 0
    for seed in range(10):
        w, prob, q, pr = _tiny_anneal_setup(40 + seed, n=7, D=2, cap=36)
        if pr["rc"] != 0:
            continue
        R = pr["r_star"]
        opt = brute.best_score(prob, w.lengths, q, R)
        an = oracle_mod.anneal(prob, w.lengths, q, R, pr["population"],
                               synth.anneal_temperatures(20), 128, seed)
        tot += 1
        hits += brute.fixed_point_to_fraction(an["best_score"], prob) == opt
    assert tot >= 5 and hits >= 0.6 * tot


@pytest.mark.parametrize("G", [1, 2])
def test_anneal_incremental_equals_full_and_nonregression(oracle_mod, G):
    w = synth.make_window("tiny", edp=G)
    prob = oracle_mod.Problem.from_dict(synth.window_problem(w))
    slot, _ = oracle_mod.place(oracle_mod.aggregate(w.demand), w.n_ranks)
    q = oracle_mod.project(w.demand, slot, w.n_ranks)
    pr = oracle_mod.pack_rows(prob, w.lengths, q, w.seed_pack, 16, 4, w.pop)
    an = oracle_mod.anneal(prob, w.lengths, q, pr["r_star"], pr["population"],
                           synth.anneal_temperatures(20), 256, w.seed_anneal, check_full=True)
    assert an["rc"] == 0
    assert tuple(an["best_score"]) <= tuple(pr["scores"].min(axis=0)) or \
        tuple(an["best_score"]) <= min(tuple(s) for s in pr["scores"])
    st, s, _, _ = oracle_mod.score(prob, w.lengths, q, pr["r_star"], an["best_layout"])
    assert st == 0 and s.tolist() == an["best_score"].tolist()


def test_anneal_resume_is_exact(oracle_mod):
    w = synth.make_window("tiny")
    prob = oracle_mod.Problem.from_dict(synth.window_problem(w))
    slot, _ = oracle_mod.place(oracle_mod.aggregate(w.demand), w.n_ranks)
    q = oracle_mod.project(w.demand, slot, w.n_ranks)
    pr = oracle_mod.pack_rows(prob, w.lengths, q, w.seed_pack, 16, 4, w.pop)
    temps = synth.anneal_temperatures(12)
    R = pr["r_star"]
    full = oracle_mod.anneal(prob, w.lengths, q, R, pr["population"], temps, 128, 77)
    a = oracle_mod.anneal(prob, w.lengths, q, R, pr["population"], temps[:5], 128, 77,
                          t_next=temps[5])
    b = oracle_mod.anneal(prob, w.lengths, q, R, a["population"], temps[5:], 128, 77,
                          sweep_offset=5, best_layout=a["best_layout"], best_score=a["best_score"])
    assert np.array_equal(full["population"], b["population"])
    assert np.array_equal(full["best_layout"], b["best_layout"])
    assert np.array_equal(full["trace"], np.concatenate([a["trace"], b["trace"]]))


def test_anneal_rejects_bad_input(oracle_mod):
    w = synth.make_window("tiny")
    prob = oracle_mod.Problem.from_dict(synth.window_problem(w))
    slot, _ = oracle_mod.place(oracle_mod.aggregate(w.demand), w.n_ranks)
    q = oracle_mod.project(w.demand, slot, w.n_ranks)
    pr = oracle_mod.pack_rows(prob, w.lengths, q, w.seed_pack, 16, 4, w.pop)
    R = pr["r_star"]
    bad = pr["population"].copy()
    bad[0, 0] = R * w.n_dp        # out-of-range cell
    assert oracle_mod.anneal(prob, w.lengths, q, R, bad, [1e-3], 8, 1)["rc"] == -4
    assert oracle_mod.anneal(prob, w.lengths, q, R, pr["population"], [1e-3, 2e-3], 8, 1)["rc"] == -1


def test_placement_load_by_hand():
    # E = 4 experts on P = 2 ranks (H = 2 slots each): identity keeps experts
    # {0, 1} on rank 0; pi = (3, 0, 1, 2) puts experts 1 and 2 there.
    agg = np.array([[5, 1, 7, 3]], dtype=np.int64)
    assert O.placement_load(agg, np.array([[0, 1, 2, 3]]), 2).tolist() == [[6, 10]]
    assert O.placement_load(agg, np.array([[3, 0, 1, 2]]), 2).tolist() == [[8, 8]]


@pytest.mark.parametrize("seed", range(6))
def test_placement_load_matches_lpt_running_loads(seed):
    """For LPT's placement the loads equal the running loads that LPT keeps
    while it places (Alg. 1), and every layer's loads sum to its aggregate."""
    rng = np.random.default_rng([19, seed])
    P = int(rng.choice([1, 2, 4, 8]))
    E = P * int(rng.integers(1, 6))
    agg = rng.integers(0, 1000, size=(3, E)).astype(np.int64)
    slot, load = O.place(agg, P)
    G = O.placement_load(agg, slot, P)
    assert np.array_equal(G, load)
    assert np.array_equal(G.sum(axis=1), agg.sum(axis=1))
    perm = np.stack([rng.permutation(E) for _ in range(3)])
    assert np.array_equal(O.placement_load(agg, perm, P).sum(axis=1), agg.sum(axis=1))
