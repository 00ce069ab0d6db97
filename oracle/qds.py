"""QualityDiversitySelect oracle -- TEST INFRASTRUCTURE ONLY.

Only tests/, the smoke check and the CPU-baseline leg of the benchmark may
import this module.  Plain numpy and Python integers, written from the
seeding passage of arXiv 2608.12146 (Sec. 4.1.1, "Diverse Fixed-Row
Seeding"; Alg. 2, the selection step before the cyclic fill; the cost
statement in Sec. 4.2).

What the paper fixes: selection starts from the exact-score winner and then
repeatedly adds the candidate maximising min_{y in P} d(x, y) - eta * delta0(x),
delta0 the normalised primary-score gap; d combines cell and row
co-assignment with a Sliced-Wasserstein sketch: the sorted projections
phi_k(x) = sort(H(x) u_k) of a normalised row-feature matrix H(x) (R* x F)
on q fixed directions u_k, compared by q^-1 sum_k ||phi_k(x) - phi_k(y)||_1 / R*.

Readings (the paper leaves these open; every value below is exact):
- Candidates arrive in (score, discovery) order, so candidate 0 is the
  exact-score winner and a lower index wins a tie.
- Row features (F = 2 + L): the row's token sum and sum of squared lengths,
  and for each MoE layer l the row's EDP-load profile sum_g max_p W(r,g,l,p).
  Each is normalised by its largest possible value (D C, D C^2 and k D C)
  and held in fixed point with QDS_FRAC fractional bits (floor).
- Directions: QDS_Q sign vectors u_k in {-1, +1}^F, bit f of Philox4x64-10
  block (counter (k, 0, 0, 4), key (seed, 0)) giving +1.
- Co-assignment: A(x, y) = number of samples whose cell holds a different
  sample set under x and y, B(x, y) the same for rows.
- d(x, y) = (A / N + B / N + E / (q R* 2^QDS_FRAC)) / 3 with
  E = sum_k ||phi_k(x) - phi_k(y)||_1; eta = 1; delta0(x) =
  (s0(x) - s0(x_0)) / s0(x_0) (0 when s0(x_0) = 0).  No quality gate.
- Every candidate is selected (the population is at least as large as the
  candidate set); the population is the selection order repeated.
"""
from __future__ import annotations

import numpy as np

from . import philox4x64

QDS_Q = 8          # projections
QDS_FRAC = 20      # fractional bits of the row features
QDS_TAG = 4        # Philox counter tag of the projection directions


def row_features(prob, lengths, q, n_rows, layout):
    """H(x): int64 [R][2 + L], the normalised row features in fixed point."""
    D, G, C, k = prob.n_dp, prob.n_edp, int(prob.capacity), int(prob.top_k)
    L, P = q.shape[1], q.shape[2]
    shard = np.asarray(prob.dp_to_edp, dtype=np.int64)
    t = np.asarray(lengths, dtype=np.int64)
    cell = np.asarray(layout, dtype=np.int64)
    row, slot = cell // D, cell % D
    H = np.zeros((n_rows, 2 + L), dtype=np.int64)
    for r in range(n_rows):
        members = np.nonzero(row == r)[0]
        T = int(t[members].sum())
        Q2 = int((t[members] ** 2).sum())
        H[r, 0] = (T << QDS_FRAC) // (D * C)
        H[r, 1] = (Q2 << QDS_FRAC) // (D * C * C)
        for l in range(L):
            E = 0
            for g in range(G):
                mg = members[shard[slot[members]] == g]
                W = q[mg, l, :].astype(np.int64).sum(axis=0) if len(mg) else np.zeros(P, np.int64)
                E += int(W.max())
            H[r, 2 + l] = (E << QDS_FRAC) // (k * D * C)
    return H


def directions(n_features, seed):
    """u_k in {-1, +1}^F from the bits of one Philox block per direction."""
    assert n_features <= 256
    U = np.empty((QDS_Q, n_features), dtype=np.int64)
    for kk in range(QDS_Q):
        blk = philox4x64([kk, 0, 0, QDS_TAG], [seed, 0])
        for f in range(n_features):
            bit = (int(blk[f // 64]) >> (f % 64)) & 1
            U[kk, f] = 1 if bit else -1
    return U


def sketch(H, U):
    """phi_k: int64 [Q][R], each projection H u_k sorted ascending."""
    return np.sort(H @ U.T, axis=0).T.copy()


def _set_changes(groups_x, groups_y):
    """Samples whose group (cell or row) holds a different sample set."""
    n = len(groups_x)
    sets_x, sets_y = {}, {}
    for i in range(n):
        sets_x.setdefault(int(groups_x[i]), []).append(i)
        sets_y.setdefault(int(groups_y[i]), []).append(i)
    changed = 0
    for i in range(n):
        if sets_x[int(groups_x[i])] != sets_y[int(groups_y[i])]:
            changed += 1
    return changed


def coassignment(prob, x, y):
    """(A, B): samples whose cell, resp. row, sample set differs."""
    x = np.asarray(x, dtype=np.int64)
    y = np.asarray(y, dtype=np.int64)
    return _set_changes(x, y), _set_changes(x // prob.n_dp, y // prob.n_dp)


def distance_numerator(prob, n_rows, x, y, phi_x, phi_y):
    """3 N q R 2^FRAC d(x, y), an integer."""
    N = len(x)
    A, B = coassignment(prob, x, y)
    E = int(np.abs(phi_x - phi_y).sum())
    return (A + B) * QDS_Q * n_rows * (1 << QDS_FRAC) + E * N


def select(prob, lengths, q, n_rows, candidates, s0, seed):
    """The selection order (a permutation of the candidates, candidate 0
    first) by the greedy max-min rule with the primary-score penalty."""
    M = len(candidates)
    N = len(lengths)
    F = 2 + q.shape[1]
    U = directions(F, seed)
    phis = [sketch(row_features(prob, lengths, q, n_rows, candidates[m]), U) for m in range(M)]
    dn = np.zeros((M, M), dtype=object)
    for a in range(M):
        for b in range(a + 1, M):
            dn[a, b] = dn[b, a] = distance_numerator(prob, n_rows, candidates[a], candidates[b], phis[a], phis[b])
    den = 3 * N * QDS_Q * n_rows * (1 << QDS_FRAC)
    sw = int(s0[0])
    order = [0]
    dmin = [dn[0, m] for m in range(M)]
    left = list(range(1, M))
    while left:
        best, best_key = None, None
        for m in left:
            # (min_y d - delta0) * den * s0(x_0), or min_y d * den when s0(x_0) = 0
            key = dmin[m] * sw - (int(s0[m]) - sw) * den if sw > 0 else dmin[m]
            if best_key is None or key > best_key:
                best, best_key = m, key
        order.append(best)
        left.remove(best)
        for m in left:
            dmin[m] = min(dmin[m], dn[best, m])
    return np.array(order, dtype=np.int32)


def population(candidates, order, pop_size):
    """P_0[m] = the candidate at order[m mod M]."""
    M = len(order)
    return np.stack([np.asarray(candidates[order[m % M]], dtype=np.int32) for m in range(pop_size)])
