"""Lower bounds on the cell count of a fixed-row layout -- TEST
INFRASTRUCTURE ONLY (only tests/, the smoke check and the CPU-baseline leg of
the benchmark may import this module).

The row count R* of Sec. 3.2 is minimal (Eq. min-row-count) when some valid
lower bound on the number of cells reaches R* D.  Besides the two bounds in
R_lb (token volume; samples longer than C/2 one per cell) this takes, on
plain definitions:
- cardinality: no cell holds k + 1 samples longer than C / (k + 1), so
  K >= ceil(#{t_i (k+1) > C} / k) for every k >= 1 (k = 1 is the C/2 bound);
- Martello and Toth's L2 (Discrete Applied Mathematics 28, 1990): for an
  integer alpha in [0, C/2], with J1 = {t > C - alpha},
  J2 = {C/2 < t <= C - alpha} and J3 = {alpha <= t <= C/2},
  K >= |J1| + |J2| + max(0, ceil((sum_J3 t - (|J2| C - sum_J2 t)) / C));
  L2 is the largest value over alpha (alpha = 0 and every t_i <= C/2).
Each bound counts bins of capacity C for the samples, so it holds for the
cells of any layout; the non-empty cells of Eq. nonempty-cell only add
constraints.
"""
from __future__ import annotations

import numpy as np


def _ceil_div(a: int, b: int) -> int:
    return -(-a // b)


def cell_lower_bound(lengths, C):
    """The largest of the volume, cardinality and L2 bounds on the cells."""
    t = np.asarray(lengths, dtype=np.int64)
    n = len(t)
    best = _ceil_div(int(t.sum()), C)
    for k in range(1, n + 1):
        best = max(best, _ceil_div(int(((k + 1) * t > C).sum()), k))
    alphas = [0] + sorted({int(v) for v in t[2 * t <= C]})
    for a in alphas:
        j1 = t > C - a
        j2 = (2 * t > C) & (t <= C - a)
        j3 = (2 * t <= C) & (t >= a)
        slack = int(j2.sum()) * C - int(t[j2].sum())
        best = max(best, int(j1.sum()) + int(j2.sum()) + max(0, _ceil_div(int(t[j3].sum()) - slack, C)))
    return best


def row_lower_bound(lengths, C, D, min_rows=1):
    """(R_bound, K_bound): R_bound = max(1, min_rows, ceil(K_bound / D))."""
    k = cell_lower_bound(lengths, C)
    return max(1, int(min_rows), _ceil_div(k, D)), k
