"""Exhaustive, exact-rational references for tiny instances -- TEST INFRASTRUCTURE.

Everything here is written straight from the paper's normalised equations with
Python Fractions, independently of the C oracle, so that it can pin it:

* score_exact: Eqs. cell-token-statistics, stage-aware-attention,
  row-expert-load, row-expert-cost and lexicographic-score (Sec. 3.4-3.5),
  with the reading that a raw-token proxy a*T + b*T2 (Eq.
  attention-cost-proxy) becomes alpha = a, beta = b*C in normalised form.
* feasible layouts by enumeration (Eqs. sample-bijection .. token-capacity)
  and the minimum row count (Eq. min-row-count).
* canonical form by its definition (Sec. 4.1.1, Canonicalize).
"""
from __future__ import annotations

import itertools
from fractions import Fraction

import numpy as np


def score_exact(prob, lengths, q, R, layout):
    """Normalised score tuple (max_g U_g, sum_g U_g, max_{r,g} J) as Fractions,
    or None when the layout is infeasible."""
    J = row_shard_costs_exact(prob, lengths, q, R, layout)
    if J is None:
        return None
    G = prob.n_edp
    U = [sum(J[(r, g)] for r in range(R)) for g in range(G)]
    return (max(U), sum(U), max(J.values()))


def row_shard_costs_exact(prob, lengths, q, R, layout):
    """J_{r,g} = A_{r,g} + E_{r,g} (Eqs. stage-aware-attention, row-expert-load,
    row-expert-cost) as Fractions keyed by (r, g), or None when the layout is
    infeasible."""
    D, G, C = prob.n_dp, prob.n_edp, prob.capacity
    L, P = prob.n_layers, prob.n_ranks
    t = [int(x) for x in lengths]
    N = len(t)
    F = 2 ** prob.frac_bits
    a = [Fraction(int(x), F) for x in prob.alpha_fp]
    b = [Fraction(int(x), F) for x in prob.beta_fp]
    cells = {c: [] for c in range(R * D)}
    for i, c in enumerate(layout):
        c = int(c)
        if c < 0 or c >= R * D:
            return None
        cells[c].append(i)
    if any(len(v) == 0 for v in cells.values()):
        return None
    if any(sum(t[i] for i in v) > C for v in cells.values()):
        return None
    Tbar = {c: Fraction(sum(t[i] for i in v), C) for c, v in cells.items()}
    Qbar = {c: sum((Fraction(t[i], C) ** 2 for i in v), Fraction(0)) for c, v in cells.items()}
    shard_slots = [[d for d in range(D) if int(prob.dp_to_edp[d]) == g] for g in range(G)]
    J = {}
    for r in range(R):
        for g in range(G):
            A = Fraction(0)
            for s in range(len(a)):
                alpha, beta = a[s], b[s] * C
                A += max(alpha * Tbar[r * D + d] + beta * Qbar[r * D + d] for d in shard_slots[g])
            E = Fraction(0)
            for l in range(L):
                W = [sum(int(q[i][l][p]) for d in shard_slots[g] for i in cells[r * D + d])
                     for p in range(P)]
                E += Fraction(max(W), C)
            J[(r, g)] = A + E
    return J


def fixed_point_to_fraction(s, prob):
    """Fixed-point score components -> normalised Fractions (divide by 2^F C)."""
    den = (2 ** prob.frac_bits) * prob.capacity
    return tuple(Fraction(int(v), den) for v in s)


def feasible_layouts(lengths, C, R, D):
    """Every assignment of samples to R*D cells with no empty cell and no cell
    over capacity (enumeration; tiny inputs only)."""
    N = len(lengths)
    K = R * D
    t = [int(x) for x in lengths]
    for assign in itertools.product(range(K), repeat=N):
        tot = [0] * K
        for i, c in enumerate(assign):
            tot[c] += t[i]
        if min(tot) == 0:
            continue  # a cell with zero tokens is empty (every t_i >= 1)
        if max(tot) > C:
            continue
        yield np.array(assign, dtype=np.int32)


def min_rows(lengths, C, D, r_hi=None):
    """Smallest R with a feasible rectangular layout (Eq. min-row-count), by
    exhaustive bin checks; None if none up to r_hi."""
    N = len(lengths)
    r_hi = N // D if r_hi is None else r_hi
    t = sorted((int(x) for x in lengths), reverse=True)
    for R in range(1, r_hi + 1):
        K = R * D
        if K > N:
            break
        if _can_pack(t, C, K):
            return R
    return None


def _can_pack(t, C, K):
    """Can items t go into exactly K non-empty bins of capacity C?"""
    bins = [0] * K
    cnt = [0] * K
    n = len(t)

    def rec(h, empty):
        if n - h < empty:
            return False
        if h == n:
            return empty == 0
        seen = set()
        for c in range(K):
            key = (bins[c], cnt[c] == 0)
            if key in seen:
                continue
            seen.add(key)
            if bins[c] + t[h] <= C:
                bins[c] += t[h]
                cnt[c] += 1
                ok = rec(h + 1, empty - (1 if cnt[c] == 1 else 0))
                bins[c] -= t[h]
                cnt[c] -= 1
                if ok:
                    return True
        return False

    return rec(0, K)


def canonical(layout, R, D, dp_to_edp):
    """Canonical form by definition: ids sorted within cells; within each
    (row, shard) the shard's cells ordered by their id tuples onto the shard's
    slots in ascending order; rows ordered by their tuple of cell tuples."""
    G = int(max(dp_to_edp)) + 1
    cells = {c: tuple(sorted(i for i, x in enumerate(layout) if int(x) == c)) for c in range(R * D)}
    rows = []
    for r in range(R):
        slots = [None] * D
        for g in range(G):
            sl = [d for d in range(D) if int(dp_to_edp[d]) == g]
            tups = sorted(cells[r * D + d] for d in sl)
            for d, tp in zip(sl, tups):
                slots[d] = tp
        rows.append(tuple(slots))
    rows.sort()
    out = np.empty(len(layout), dtype=np.int32)
    for nr, row in enumerate(rows):
        for d, tp in enumerate(row):
            for i in tp:
                out[i] = nr * D + d
    return out


def best_score(prob, lengths, q, R):
    """Exact optimum (lexicographic) over all feasible layouts with R rows."""
    best = None
    for lay in feasible_layouts(lengths, prob.capacity, R, prob.n_dp):
        s = score_exact(prob, lengths, q, R, lay)
        if s is not None and (best is None or s < best):
            best = s
    return best
