"""Exact fixed-bin feasibility search -- TEST INFRASTRUCTURE ONLY (only
tests/, the smoke check and the CPU-baseline leg of the benchmark may import
this module).

Decides whether the fixed-row feasible set X_R of Sec. 3.2 is non-empty
(Eqs. sample-bijection, nonempty-cell and token-capacity with K = R D cells)
by depth-first branch and bound under a node budget, the "fixed-bin
feasibility check" the paper runs under a planning-time limit.  The search
order is fixed so that any implementation of it visits the same nodes:
- samples in (-t, i) order; sample h goes to an open cell with room, lowest
  index first, then to a new cell (the first unopened one: unopened cells
  are interchangeable);
- a sample whose length equals the previous sample's goes to no lower cell
  than that sample did (equal samples are interchangeable);
- a node is one placement; the search stops when K cells are open and all
  samples placed (feasible), when the tree is exhausted (infeasible), or
  after the budget of placements (unknown);
- a branch is cut when fewer samples remain than cells still unopened.
Returns (status, nodes, cell of each sample): status 1 feasible, 0
infeasible, 2 unknown; the cells are those of the first solution found.
"""
from __future__ import annotations

import numpy as np

FEASIBLE, INFEASIBLE, UNKNOWN = 1, 0, 2


def search(lengths, C, K, budget):
    t = np.asarray(lengths, dtype=np.int64)
    n = len(t)
    order = sorted(range(n), key=lambda i: (-int(t[i]), i))
    ts = [int(t[i]) for i in order]
    if K < 1 or K > n or max(ts) > C:
        return INFEASIBLE, 0, None
    load = [0] * K
    choice = [-1] * n
    opened = 0
    nodes = 0
    h = 0
    while True:
        if h == n:  # every sample placed; the cut leaves no cell unopened
            cells = np.empty(n, dtype=np.int32)
            for u in range(n):
                cells[order[u]] = choice[u]
            return FEASIBLE, nodes, cells
        else:
            # the next cell for sample h after choice[h]
            lo = choice[h] + 1
            if choice[h] < 0 and h > 0 and ts[h] == ts[h - 1]:
                lo = choice[h - 1]
            b = -1
            for c in range(lo, opened):
                if load[c] + ts[h] <= C:
                    b = c
                    break
            if b < 0 and lo <= opened < K:
                b = opened
            if b >= 0:
                nodes += 1
                if nodes > budget:
                    return UNKNOWN, nodes - 1, None
                if b == opened:
                    opened += 1
                load[b] += ts[h]
                choice[h] = b
                if n - (h + 1) >= K - opened:
                    h += 1
                    if h < n:
                        choice[h] = -1
                    continue
                # cut: undo and try the next cell for h
                load[b] -= ts[h]
                if load[b] == 0:
                    opened -= 1
                continue
        # backtrack: sample h has no cell left
        choice[h] = -1
        h -= 1
        if h < 0:
            return INFEASIBLE, nodes, None
        b = choice[h]
        load[b] -= ts[h]
        if load[b] == 0:
            opened -= 1
