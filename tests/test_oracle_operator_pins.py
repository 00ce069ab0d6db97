"""Pins of the oracle's seeding operators (Sec. 4.1.1), GuidedProposal
(Sec. 4.1.2), the energy and accept test (Eq. pa-energy, Alg. 3), the tie
rules of the trajectory best and the incumbent (Alg. 3), and the load
diagnostics (Sec. 5.3, Eqs. global-ep-cv and ep-efficiency).

None of these compares the oracle with itself.  Expected values come from
hand traces written out beside each case, random words from
numpy.random.Philox (block c of the counter-based generator is numpy's block
after counter c - 1), row-shard costs from exact rationals
(oracle/brute.py, written from the normalised equations), and diagnostics
from numpy.  Each case is built so that a plausible slip in the oracle (a key
order swapped, a roulette made uniform, a coefficient moved, a tie rule
loosened, a variance for a deviation) changes the result.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle as O
from oracle import brute

M64 = (1 << 64) - 1
P_GUIDE = 0xCCCCCCCD
RHO = 0x40000000


def philox_block(counter, key):
    """Philox4x64-10 block at a 4-word counter (word 0 least significant),
    from numpy.random.Philox, which increments its counter before a block."""
    c = sum(int(w) << (64 * k) for k, w in enumerate(counter))
    prev = (c - 1) % (1 << 256)
    words = np.array([(prev >> (64 * k)) & M64 for k in range(4)], dtype=np.uint64)
    gen = np.random.Philox(key=np.array([int(key[0]), int(key[1])], dtype=np.uint64), counter=words)
    return [int(x) for x in gen.random_raw(4)]


def bnd(w, m):
    """Bounded draw floor(w m / 2^64)."""
    return (int(w) * int(m)) >> 64


def seed_word(seed, draw, trial, phase):
    return philox_block([draw, trial, phase, 3], [seed, 0])[0]


def step_words(seed, level, replica, k=0):
    return (philox_block([k, level, replica, 0], [seed, 0]) +
            philox_block([k, level, replica, 1], [seed, 0]))


def _problem(N, L, P, D, G, dp_to_edp, C, alpha=(4096,), beta=(1,)):
    return O.Problem(N, L, P, 1, P, D, G, dp_to_edp, C, list(alpha), list(beta))


# --------------------------------------------------------------------------
# WindowShuffle (Sec. 4.1.1): repeatedly take one of the first w remaining
# samples of the (-t, i) order.
def test_window_shuffle_width_one_keeps_length_order():
    t = np.array([5, 9, 9, 1, 7, 3, 7, 2], dtype=np.int32)
    prob = _problem(8, 1, 2, 2, 1, [0, 0], 100)
    q = np.zeros((8, 1, 2), dtype=np.int32)
    for trial in (0, 1, 5):
        r = O.seed_trial(prob, t, q, 2, 1, 91, trial)
        # (-t, i): 9(1), 9(2), 7(4), 7(6), 5(0), 3(5), 2(7), 1(3)
        assert r["pi"].tolist() == [1, 2, 4, 6, 0, 5, 7, 3]


@pytest.mark.parametrize("seed,trial", [(91, 0), (91, 3), (7, 1), (2608, 2)])
def test_window_shuffle_width_two_follows_the_word_top_bit(seed, trial):
    """With w = 2 a bounded draw over two positions is the top bit of the
    word: the next sample is the first remaining one when the bit is 0."""
    t = np.array([5, 9, 9, 1, 7, 3, 7, 2, 4, 6], dtype=np.int32)
    prob = _problem(10, 1, 2, 2, 1, [0, 0], 100)
    q = np.zeros((10, 1, 2), dtype=np.int32)
    r = O.seed_trial(prob, t, q, 2, 2, seed, trial)
    rem = [1, 2, 4, 6, 9, 0, 8, 5, 7, 3]            # the (-t, i) order
    bits = [seed_word(seed, h, trial, 0) >> 63 for h in range(10)]
    assert 0 < sum(bits[:9]) < 9                      # both branches are exercised
    want = []
    for h in range(10):
        want.append(rem.pop(bits[h] if len(rem) >= 2 else 0))
    assert r["pi"].tolist() == want


# --------------------------------------------------------------------------
# RandomizedBestFit (Sec. 4.1.1): feasible cells ranked by decreasing token
# occupancy, then ascending cardinality, then ascending index.
def test_best_fit_prefers_fewer_members_on_equal_occupancy():
    # t = (8, 6, 2, 1), C = 9, K = 2 cells.  Samples 0 and 1 open cells 0 and
    # 1.  Sample 2 (t = 2) fits only cell 1 (8 + 2 > 9): cell 1 = {1, 2},
    # T = 8.  Sample 3 (t = 1) fits both; both hold 8 tokens, cell 0 has one
    # member and cell 1 two, so cell 0 takes it.
    prob = _problem(4, 1, 2, 1, 1, [0], 9)
    q = np.zeros((4, 1, 2), dtype=np.int32)
    r = O.seed_trial(prob, np.array([8, 6, 2, 1], dtype=np.int32), q, 2, 1, 5, 0)
    assert r["ok"] and r["cellk"].tolist() == [0, 1, 1, 0]


def test_best_fit_occupancy_then_index():
    # t = (5, 5, 3, 1), C = 9.  Cells 0 = {0} and 1 = {1} tie on T and size,
    # so sample 2 goes to the lower index (cell 0, T = 8).  Sample 3 then goes
    # to the fuller cell 0 (8 > 5), which it fills exactly.
    prob = _problem(4, 1, 2, 1, 1, [0], 9)
    q = np.zeros((4, 1, 2), dtype=np.int32)
    r = O.seed_trial(prob, np.array([5, 5, 3, 1], dtype=np.int32), q, 2, 1, 5, 0)
    assert r["ok"] and r["cellk"].tolist() == [0, 1, 0, 0]


def test_best_fit_reports_a_dead_end():
    # t = (6, 6, 5), C = 10, K = 2: the 5 fits neither cell.
    prob = _problem(3, 1, 2, 1, 1, [0], 10)
    q = np.zeros((3, 1, 2), dtype=np.int32)
    assert not O.seed_trial(prob, np.array([6, 6, 5], dtype=np.int32), q, 2, 1, 5, 0)["ok"]


@pytest.mark.parametrize("w,seed", [(2, 3), (3, 4), (4, 11)])
def test_best_fit_rank_is_the_bounded_draw(w, seed):
    """Each sample after the first K takes the feasible cell at rank
    bnd(word, min(w, |F|)) of the (-T, size, index) order."""
    rng = np.random.default_rng([7, w, seed])
    N, D, R, C = 24, 2, 3, 60
    t = rng.integers(1, 16, size=N).astype(np.int32)
    prob = _problem(N, 1, 2, D, 1, [0, 0], C)
    q = np.zeros((N, 1, 2), dtype=np.int32)
    trial = 2
    r = O.seed_trial(prob, t, q, R, w, seed, trial)
    assert r["ok"]
    K = R * D
    T, n = [0] * K, [0] * K
    ranks = []
    for h, i in enumerate(r["pi"].tolist()):
        if h < K:
            assert r["cellk"][i] == h
            T[h], n[h] = int(t[i]), 1
            continue
        F = sorted((c for c in range(K) if T[c] + int(t[i]) <= C), key=lambda c: (-T[c], n[c], c))
        rho = bnd(seed_word(seed, h, trial, 1), min(w, len(F)))
        ranks.append(rho)
        c = F[rho]
        assert r["cellk"][i] == c, h
        T[c] += int(t[i])
        n[c] += 1
    assert len(set(ranks)) > 1


# --------------------------------------------------------------------------
# EDPAwarePair (Sec. 4.1.1): cells by decreasing routed peak sum_l max_p Q,
# each into the row-shard with room minimising (increase of sum_l max_p W,
# resulting max W, r, g); the cell takes the lowest empty slot of D_g.
def test_edp_pair_prefers_the_smaller_increase():
    # L = 2, P = 2, D = 2, G = 1, R = 2; one sample per cell.
    #   cell 0: [[10, 0], [0, 0]]  peak 10
    #   cell 1: [[0, 9], [0, 0]]   peak 9
    #   cell 2: [[0, 0], [4, 4]]   peak 4
    #   cell 3: [[1, 1], [1, 1]]   peak 2
    # Cell 0 ties on both rows (increase 10, max 10) -> row 0, slot 0.
    # Cell 1: row 0 gives increase 0 and max 10, row 1 increase 9 and max 9;
    # the increase decides -> row 0, slot 1.  Cells 2 and 3 fill row 1.
    q = np.array([[[10, 0], [0, 0]], [[0, 9], [0, 0]], [[0, 0], [4, 4]], [[1, 1], [1, 1]]],
                 dtype=np.int32)
    prob = _problem(4, 2, 2, 2, 1, [0, 0], 100)
    lay = O.edp_pair(prob, q, 2, np.array([0, 1, 2, 3]), 1, 1, 0)
    assert lay.tolist() == [0, 1, 2, 3]


def test_edp_pair_peak_order_and_shard_slots():
    # L = 1, P = 2, D = 4, G = 2 with slots D_0 = {0, 2} and D_1 = {1, 3}; R = 1.
    #   cell 0: [2, 0] peak 2;  cell 1: [0, 5] peak 5;  cell 2: [5, 0] peak 5;
    #   cell 3: [0, 1] peak 1.  Visit order (-peak, c): 1, 2, 0, 3.
    # Cell 1 ties everywhere -> (r, g) = (0, 0), slot 0.  Cell 2: shard 0
    # gives increase 0 ([5, 5]), shard 1 increase 5 -> shard 0, slot 2.
    # Shard 0 is full: cell 0 -> slot 1, cell 3 -> slot 3.
    q = np.array([[[2, 0]], [[0, 5]], [[5, 0]], [[0, 1]]], dtype=np.int32)
    prob = _problem(4, 1, 2, 4, 2, [0, 1, 0, 1], 100)
    lay = O.edp_pair(prob, q, 1, np.array([0, 1, 2, 3]), 1, 1, 0)
    assert lay.tolist() == [1, 0, 2, 3]


def test_edp_pair_resulting_max_breaks_increase_ties():
    # L = 1, P = 2, D = 2, G = 1, R = 2; one sample per cell.
    #   cell 0: [4, 0] peak 4 -> both rows tie -> row 0, slot 0.
    #   cell 1: [3, 0] peak 3: row 0 gives increase 3 and max 7, row 1
    #           increase 3 and max 3; the smaller max picks row 1, slot 0.
    #   cell 2: [1, 0] peak 1: row 0 -> increase 1, max 5; row 1 -> increase
    #           1, max 4 -> row 1, slot 1.
    #   cell 3: [0, 1] peak 1 (after cell 2 by index): only row 0 has room.
    q = np.array([[[4, 0]], [[3, 0]], [[1, 0]], [[0, 1]]], dtype=np.int32)
    prob = _problem(4, 1, 2, 2, 1, [0, 0], 100)
    lay = O.edp_pair(prob, q, 2, np.array([0, 1, 2, 3]), 1, 1, 0)
    assert lay.tolist() == [0, 2, 3, 1]


@pytest.mark.parametrize("w,seed,G", [(2, 5, 1), (3, 6, 1), (2, 8, 2), (4, 9, 2)])
def test_edp_pair_rank_draw_weights(w, seed, G):
    """The rank among the leading w' = min(w, #candidates) is drawn with
    weights 2^(w' - 1 - rank) by a roulette on bnd(word, 2^w' - 1)."""
    rng = np.random.default_rng([8, w, seed, G])
    L, P, D, R = 3, 4, 4, 3
    dp = [0, 0, 0, 0] if G == 1 else [0, 1, 0, 1]
    K = R * D
    q = rng.integers(0, 20, size=(K, L, P)).astype(np.int32)
    prob = _problem(K, L, P, D, G, dp, 1000)
    trial = 3
    lay = O.edp_pair(prob, q, R, np.arange(K), w, seed, trial)
    slots = [[d for d in range(D) if dp[d] == g] for g in range(G)]
    peak = q.max(axis=2).sum(axis=1)
    order = sorted(range(K), key=lambda k: (-int(peak[k]), k))
    Wt = np.zeros((R * G, L, P), dtype=np.int64)
    filled = [0] * (R * G)
    rhos = []
    for pos, k in enumerate(order):
        cands = []
        for h in range(R * G):
            if filled[h] >= len(slots[h % G]):
                continue
            after = Wt[h] + q[k]
            inc = int(after.max(axis=1).sum() - Wt[h].max(axis=1).sum())
            cands.append((inc, int(after.max()), h // G, h % G))
        cands.sort()
        wp = min(w, len(cands))
        pick = bnd(seed_word(seed, pos, trial, 2), (1 << wp) - 1)
        rho, pref = 0, 0
        for rho in range(wp):
            pref += 1 << (wp - 1 - rho)
            if pref > pick:
                break
        rhos.append(rho)
        _, _, r, g = cands[rho]
        h = r * G + g
        d = slots[g][filled[h]]
        filled[h] += 1
        Wt[h] += q[k]
        assert lay[k] == r * D + d, pos
    assert len(set(rhos)) > 1


# --------------------------------------------------------------------------
# GuidedProposal (Sec. 4.1.2) and the random branch: one step per member at an
# infinite temperature accepts every feasible proposal, so each member's
# terminal layout shows the proposal its replica's words made.
def _guided_instance(G):
    rng = np.random.default_rng([31, G])
    N, L, P, D, R = 16, 2, 2, 4, 2
    dp = [0, 0, 0, 0] if G == 1 else [0, 0, 1, 1]
    t = rng.integers(10, 200, size=N).astype(np.int32)
    t[:4] = [900, 700, 30, 20]          # skewed rows: J and cell costs far apart
    q = rng.integers(0, 200, size=(N, L, P)).astype(np.int32)
    q[:4] *= 5
    lay = np.arange(N, dtype=np.int32) % (R * D)
    lay[[0, 1, 2, 3]] = [0, 1, 0, 1]    # the long samples share row 0
    lay[[4, 5]] = [2, 3]
    prob = _problem(N, L, P, D, G, dp, 4096, alpha=(4096, 2048), beta=(0, 1))
    return prob, t, q, R, lay


def _predict_step(prob, t, q, R, lay, words):
    """The proposal of one step (Sec. 4.1.2 with the readings of the
    deterministic spec) -> (i, j or -1, source cell, target cell, guided)."""
    N, D, G = prob.n_samples, prob.n_dp, prob.n_edp
    dp = [int(x) for x in prob.dp_to_edp]
    slots = [[d for d in range(D) if dp[d] == g] for g in range(G)]
    F = 2 ** prob.frac_bits
    Cp = prob.capacity
    cells = {c: sorted(i for i in range(N) if lay[i] == c) for c in range(R * D)}
    Jf = brute.row_shard_costs_exact(prob, t, q, R, lay)
    J = []
    for h in range(R * G):
        v = Jf[(h // G, h % G)] * F * Cp
        assert v.denominator == 1
        J.append(int(v))
    w = words
    guided = (w[0] & 0xFFFFFFFF) < P_GUIDE
    reloc = (w[0] >> 32) < RHO

    def roulette(wts, word):
        tot = sum(wts)
        if tot == 0:
            return bnd(word, len(wts))
        return int(np.searchsorted(np.cumsum(wts), bnd(word, tot), side="right"))

    if guided:
        h1 = roulette(J, w[1])
        r1, g1 = divmod(h1, G)
        costs = []
        for d in slots[g1]:
            Tc = sum(int(t[i]) for i in cells[r1 * D + d])
            Qc = sum(int(t[i]) ** 2 for i in cells[r1 * D + d])
            costs.append(sum(int(a) * Tc + int(b) * Qc for a, b in zip(prob.alpha_fp, prob.beta_fp)))
        ca = r1 * D + slots[g1][roulette(costs, w[2])]
        i = cells[ca][bnd(w[3], len(cells[ca]))]
        jmax = max(J)
        h2 = roulette([jmax - x + 1 for x in J], w[4])
        r2, g2 = divmod(h2, G)
        cb = r2 * D + slots[g2][bnd(w[5], len(slots[g2]))]
        j = -1 if reloc else cells[cb][bnd(w[6], len(cells[cb]))]
    else:
        i = bnd(w[1], N)
        ca = int(lay[i])
        if reloc:
            j, cb = -1, bnd(w[4], R * D)
        else:
            j = bnd(w[4], N)
            cb = int(lay[j])
    return i, j, ca, cb, guided


def _apply(prob, t, lay, i, j, ca, cb):
    """Layout after the move, or None when it is infeasible (Alg. 3: equal
    cells, a cell over capacity, or a relocation that empties its cell)."""
    if ca == cb:
        return None
    T = np.bincount(lay, weights=t, minlength=int(lay.max()) + 1)
    n = np.bincount(lay, minlength=int(lay.max()) + 1)
    tj = int(t[j]) if j >= 0 else 0
    if j >= 0:
        if T[ca] - t[i] + tj > prob.capacity or T[cb] - tj + t[i] > prob.capacity:
            return None
    elif n[ca] < 2 or T[cb] + t[i] > prob.capacity:
        return None
    out = lay.copy()
    out[i] = cb
    if j >= 0:
        out[j] = ca
    return out


@pytest.mark.parametrize("G", [1, 2])
def test_guided_proposal_roulettes(G):
    prob, t, q, R, lay = _guided_instance(G)
    pop, seed = 192, 4242
    an = O.anneal(prob, t, q, R, np.tile(lay, (pop, 1)), [1e300], 1, seed,
                  replica_ids=np.arange(pop), want_steps=True)
    assert an["rc"] == 0
    n_guided = n_moved = 0
    for j in range(pop):
        i, jj, ca, cb, guided = _predict_step(prob, t, q, R, lay, step_words(seed, 0, j))
        want = _apply(prob, t, lay, i, jj, ca, cb)
        n_guided += guided
        if want is None:
            assert an["steps"][0, j, 0] == 0 and np.array_equal(an["population"][j], lay), j
        else:
            n_moved += 1
            assert an["steps"][0, j, 0] == 2 and np.array_equal(an["population"][j], want), j
    assert n_guided > pop // 2 and n_moved > pop // 3


# --------------------------------------------------------------------------
# Energy (Eq. pa-energy) and the accept test (Alg. 3): an uphill step is
# accepted iff u < exp(-Delta / T) with Delta = (E' - E) / max(|E|, 1).  The
# temperature threshold of a known step is T* = Delta / (-ln u): a step at
# 1.05 T* must be accepted and one at T* / 1.05 rejected.
def _energy(s):
    S = [float(x) for x in s]
    return (S[0] + 1e-6 * S[1]) + 1e-9 * S[2]


def _uphill_steps(prob, t, q, R, lay, seed, n_replicas):
    s0 = brute.score_exact(prob, t, q, R, lay)
    out = []
    for rid in range(n_replicas):
        w = step_words(seed, 0, rid)
        i, j, ca, cb, _ = _predict_step(prob, t, q, R, lay, w)
        nl = _apply(prob, t, lay, i, j, ca, cb)
        if nl is None:
            continue
        s1 = brute.score_exact(prob, t, q, R, nl)
        if not s1 > s0:
            continue
        u = (w[7] >> 32) / 2.0**32
        if not 0.05 < u < 0.95:
            continue
        e0, e1 = _energy(s0), _energy(s1)
        out.append(dict(rid=rid, s0=s0, s1=s1, u=u, delta=(e1 - e0) / max(abs(e0), 1.0), e0=e0))
    return out


def _check_threshold(prob, t, q, R, lay, seed, st):
    tstar = st["delta"] / -math.log(st["u"])
    for temp, code in ((tstar * 1.05, 2), (tstar / 1.05, 1)):
        an = O.anneal(prob, t, q, R, lay[None, :], [temp], 1, seed, replica_ids=[st["rid"]],
                      want_steps=True)
        assert an["rc"] == 0 and an["steps"][0, 0, 0] == code, (st, temp)


def test_accept_threshold_with_the_max_shard_unchanged():
    """Two EDP shards, a step inside the lighter shard: S0 is unchanged, S1
    rises, so the step's Delta is carried by the 1e-6 weight of S1 (the 1e-9
    weight belongs to S2); |E| > 1 so the max(|E|, 1) scale is |E|."""
    prob, t, q, R, lay = _guided_instance(2)
    seed = 77
    steps = _uphill_steps(prob, t, q, R, lay, seed, 600)
    pick = [s for s in steps if s["s1"][0] == s["s0"][0] and s["s1"][1] != s["s0"][1]
            and s["s1"][2] == s["s0"][2]]
    assert pick and pick[0]["e0"] > 1.5
    _check_threshold(prob, t, q, R, lay, seed, pick[0])
    pick2 = [s for s in steps if s["s1"][0] > s["s0"][0]]
    assert pick2
    _check_threshold(prob, t, q, R, lay, seed, pick2[0])


def test_accept_threshold_below_unit_energy():
    """|E| < 1: Delta is the raw energy difference (max(|E|, 1) = 1)."""
    N, D, R = 8, 2, 2
    t = np.array([30, 25, 20, 18, 12, 9, 7, 5], dtype=np.int32)
    prob = _problem(N, 0, 2, D, 1, [0, 0], 1000, alpha=(4096,), beta=(0,))
    q = np.zeros((N, 0, 2), dtype=np.int32)
    lay = np.array([0, 1, 2, 3, 0, 1, 2, 3], dtype=np.int32)
    seed = 5
    steps = _uphill_steps(prob, t, q, R, lay, seed, 400)
    assert steps and steps[0]["e0"] < 0.5
    _check_threshold(prob, t, q, R, lay, seed, steps[0])


# --------------------------------------------------------------------------
# Tie rules (Alg. 3): the trajectory best and the incumbent change only on a
# strict lexicographic improvement, members scanned in ascending order.
def _twin_instance():
    # Four samples of equal length and equal routing: every layout with two
    # samples per cell has the same score, and the layouts differ.
    t = np.array([4, 4, 4, 4], dtype=np.int32)
    q = np.ones((4, 1, 2), dtype=np.int32)
    prob = _problem(4, 1, 2, 2, 1, [0, 0], 12)
    return prob, t, q


def test_incumbent_keeps_the_first_of_equal_members():
    prob, t, q = _twin_instance()
    a = np.array([0, 0, 1, 1], dtype=np.int32)
    b = np.array([0, 1, 0, 1], dtype=np.int32)
    assert brute.score_exact(prob, t, q, 1, a) == brute.score_exact(prob, t, q, 1, b)
    # K = 0: each member's trajectory best is its start state.
    an = O.anneal(prob, t, q, 1, np.stack([a, b]), [1.0], 0, 3)
    assert an["rc"] == 0 and an["best_layout"].tolist() == a.tolist()
    # A given incumbent of equal score is kept against both members.
    st, s, _, _ = O.score(prob, t, q, 1, b)
    an = O.anneal(prob, t, q, 1, np.stack([a, b]), [1.0], 0, 3, best_layout=b, best_score=s)
    assert an["rc"] == 0 and an["best_layout"].tolist() == b.tolist()
    # A worse given incumbent is replaced by member 0, not member 1.
    worse = np.array([0, 0, 0, 1], dtype=np.int32)
    st, sw, _, _ = O.score(prob, t, q, 1, worse)
    assert st == 0 and tuple(sw) > tuple(s)
    an = O.anneal(prob, t, q, 1, np.stack([a, b]), [1.0], 0, 3, best_layout=worse, best_score=sw)
    assert an["rc"] == 0 and an["best_layout"].tolist() == a.tolist()


def test_trajectory_best_keeps_the_first_of_equal_states():
    """Near zero temperature only improving or equal moves pass; from an
    optimal start the chain walks among equal-score layouts (swaps of twins),
    and its trajectory best must stay the start layout."""
    prob, t, q = _twin_instance()
    start = np.array([0, 0, 1, 1], dtype=np.int32)
    worse = np.array([0, 0, 0, 1], dtype=np.int32)
    st, sw, _, _ = O.score(prob, t, q, 1, worse)
    an = O.anneal(prob, t, q, 1, start[None, :], [1e-300], 64, 12, best_layout=worse, best_score=sw,
                  want_steps=True)
    assert an["rc"] == 0
    assert (an["steps"][0, 0] == 2).sum() >= 2            # equal swaps were accepted
    assert not np.array_equal(an["population"][0], start)  # and moved the chain
    assert an["best_layout"].tolist() == start.tolist()


# --------------------------------------------------------------------------
# Load diagnostics (Sec. 5.3): CV_global (Eq. global-ep-cv) from the window
# rank loads; S_EP, T_EP and eta_EP (Eq. ep-efficiency) from the row loads.
def test_diagnostics_on_the_fig3_instance():
    # Fig. 3: identity placement gives window loads 12 vs 4 (CV 0.5, row peaks
    # 6); LPT gives 8 vs 8 (CV 0).  Under LPT, {A,B}{C,D} has row peaks 8 and
    # 8 with means 4 and 4 (eta 0.5); {A,C}{B,D} has peaks 4 and 4 (eta 1).
    demand = np.array([[[3, 0, 1, 0]], [[3, 0, 1, 0]], [[0, 3, 0, 1]], [[0, 3, 0, 1]]], dtype=np.int32)
    t = [4, 4, 4, 4]
    prob = O.Problem(4, 1, 4, 1, 2, 1, 1, [0], 8, [4096], [0])
    ident = np.arange(4, dtype=np.int32)[None, :]
    q_id = O.project(demand, ident, 2)
    st, _, _, dg = O.score(prob, t, q_id, 2, [0, 0, 1, 1], rank_load=[[12, 4]], want_diag=True)
    assert st == 0 and dg[0] == 0.5 and dg[1] == 12 and dg[2] == 6
    assert dg[3] == pytest.approx(8 / 12, rel=1e-15)
    slot, load = O.place(O.aggregate(demand), 2)
    q = O.project(demand, slot, 2)
    for lay, s_ep, t_ep, eta in (([0, 0, 1, 1], 16, 8, 0.5), ([0, 1, 0, 1], 8, 4, 1.0)):
        st, _, _, dg = O.score(prob, t, q, 2, lay, rank_load=load, want_diag=True)
        assert st == 0 and dg[0] == 0.0 and (dg[1], dg[2], dg[3]) == (s_ep, t_ep, eta)


@pytest.mark.parametrize("seed,G", [(0, 1), (1, 2), (2, 2), (3, 4)])
def test_diagnostics_match_numpy(seed, G):
    rng = np.random.default_rng([41, seed, G])
    L, P, D, R = 3, 4, 4, 3
    N = 40
    dp = np.repeat(np.arange(G), D // G).astype(np.int32)
    t = rng.integers(1, 50, size=N).astype(np.int32)
    q = rng.integers(0, 30, size=(N, L, P)).astype(np.int32)
    lay = rng.permutation(np.arange(N) % (R * D)).astype(np.int32)
    rank_load = rng.integers(1, 10**6, size=(L, P)).astype(np.int64)
    prob = O.Problem(N, L, P, 1, P, D, G, dp, 10**4, [4096, 100], [3, 1])
    st, s, J, dg = O.score(prob, t, q, R, lay, rank_load=rank_load, want_J=True, want_diag=True)
    assert st == 0
    mean = rank_load.mean(axis=1)
    cv = float(np.mean(rank_load.std(axis=1) / mean))
    W = np.zeros((R, G, L, P), dtype=np.int64)
    np.add.at(W, (lay // D, dp[lay % D]), q)
    s_ep = W.max(axis=(1, 3)).sum()
    t_ep = W.max()
    eta = W.mean(axis=3).max(axis=1).sum() / s_ep
    scale = 4096.0 * 10**4
    A = J.reshape(R, G) - (W.max(axis=3).sum(axis=2) << 12)
    assert dg[0] == pytest.approx(cv, rel=1e-12)
    assert (dg[1], dg[2]) == (s_ep, t_ep)
    assert dg[3] == pytest.approx(eta, rel=1e-12)
    assert dg[4] == pytest.approx(A.sum() / scale, rel=1e-12)
    S = s / scale
    assert (dg[5], dg[6]) == (S[0], S[1])
    assert dg[7] == (S[0] + 1e-6 * S[1]) + 1e-9 * S[2]


def test_guided_target_weight_keeps_the_heaviest_row_shard():
    """With unit fixed-point scale (F = 0) the row-shard costs are small
    integers, so the + 1 of the target weights J_max - J + 1 (which gives the
    heaviest row-shard a chance of being a target) changes picks."""
    rng = np.random.default_rng(57)
    N, L, P, D, R = 12, 1, 2, 2, 3
    t = rng.integers(1, 7, size=N).astype(np.int32)
    q = rng.integers(0, 4, size=(N, L, P)).astype(np.int32)
    prob = O.Problem(N, L, P, 1, P, D, 1, [0, 0], 100, [1], [0], frac_bits=0)
    lay = (np.arange(N) % (R * D)).astype(np.int32)
    J = brute.row_shard_costs_exact(prob, t, q, R, lay)
    Jv = sorted(int(J[(r, 0)] * 100) for r in range(R))
    assert Jv[-1] - Jv[0] <= 8                     # weights of a few units each
    pop, seed = 256, 9
    an = O.anneal(prob, t, q, R, np.tile(lay, (pop, 1)), [1e300], 1, seed,
                  replica_ids=np.arange(pop), want_steps=True)
    assert an["rc"] == 0
    for j in range(pop):
        i, jj, ca, cb, guided = _predict_step(prob, t, q, R, lay, step_words(seed, 0, j))
        want = _apply(prob, t, lay, i, jj, ca, cb)
        got = an["population"][j]
        assert np.array_equal(got, lay if want is None else want), j


# --------------------------------------------------------------------------
# Systematic resampling (Alg. 3, level boundary; Carpenter, Clifford and
# Fearnhead 1999) for a given uniform: u_m = (V / 2^32 + m) / P and member m
# takes the first j with F_j / F_{P-1} >= u_m.
def test_resample_literal_boundary_at_zero_uniform():
    # Equal weights and V = 0: F_j / F_{P-1} = (j + 1) / P >= m / P first holds
    # at j = max(m - 1, 0), so members 0 and 1 both take parent 0.
    assert O.resample_at(np.zeros(6), 1e-3, 5e-4, 0).tolist() == [0, 0, 1, 2, 3, 4]
    # With V > 0 equal weights give the identity.
    assert O.resample_at(np.zeros(6), 1e-3, 5e-4, 12345).tolist() == [0, 1, 2, 3, 4, 5]


@pytest.mark.parametrize("seed", range(6))
def test_resample_matches_real_systematic_resampling(seed):
    """Weights exp(-(1/T_next - 1/T_cur) E~_j) with E~_j = (E_j - E_min) /
    max(|E_min|, 1), from math.exp; members whose u_m lies within 1e-9 of a
    cumulative weight are skipped (there the quantised weights decide)."""
    rng = np.random.default_rng([23, seed])
    P = int(rng.integers(5, 60))
    emin = float(rng.choice([0.3, 2.5, 40.0]))
    E = emin + rng.uniform(0, 3e-4, size=P) * max(abs(emin), 1.0)
    E[int(rng.integers(P))] = emin
    t_cur, t_next = 1e-4, 6e-5
    V = int(rng.integers(0, 2**32))
    par = O.resample_at(E, t_cur, t_next, V)
    c = 1 / t_next - 1 / t_cur
    wts = [math.exp(-(c * ((e - emin) / max(abs(emin), 1.0)))) for e in E]
    F = np.cumsum(wts) / sum(wts)
    checked = 0
    for m in range(P):
        u = (V / 2.0**32 + m) / P
        if np.min(np.abs(F - u)) < 1e-9:
            continue
        assert par[m] == int(np.argmax(F >= u)), m
        checked += 1
    assert checked >= P - 2
    assert len(set(par.tolist())) < P              # some members were dropped
