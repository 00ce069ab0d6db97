"""Parity of the synthetic planner comparison (bench.py --compare): the
identity placement's rank loads and projection, the FFD layout, the annealed
incumbent and every planner's diagnostics equal the oracle's (layouts and
integer results exactly, float diagnostics to a relative 1e-6); plus the
projection entry point on its own, against the oracle, and its errors."""
import numpy as np
import pytest

import synth

gpu = pytest.mark.gpu


def _log(msg):
    print(f"[gpu-compare] {msg}", flush=True)


@gpu
@pytest.mark.parametrize("name,levels", [("tiny", None), ("small", 3)])
def test_planner_comparison_matches_oracle(name, levels):
    import bench
    import oracle as O
    import paper_2608_12146_amd as rp
    from synth import windows as W
    w = synth.make_window(name)
    pd = synth.window_problem(w)
    levels = levels or w.levels
    _log(f"compare {name}: levels {levels}")
    got = bench.compare_planners(rp, w, pd, levels)
    pb = O.Problem.from_dict(pd)
    P = w.n_ranks
    agg = O.aggregate(w.demand)
    ident = np.tile(np.arange(w.n_experts, dtype=np.int32), (w.n_layers, 1))
    q_id, g_id = O.project(w.demand, ident, P), O.placement_load(agg, ident, P)
    slot, g = O.place(agg, P)
    q = O.project(w.demand, slot, P)
    f = O.pack_rows(pb, w.lengths, q, w.seed_pack, 2, 1, 2)
    R = f["r_star"]
    x_ffd = f["population"][f["n_distinct"] - 1]
    pr = O.pack_rows(pb, w.lengths, q, w.seed_pack, W.N_TRIALS, W.CHOICE_WIDTH, w.pop)
    temps = synth.anneal_temperatures(w.levels)[:levels]
    _log(f"compare {name}: oracle annealing")
    oa = O.anneal(pb, w.lengths, q, R, pr["population"], temps, W.STEPS_PER_LEVEL, w.seed_anneal,
                  want_trace=False, want_parents=False)
    assert oa["rc"] == 0
    assert got["n_rows"] == R
    assert np.array_equal(got["layouts"]["ffd"], x_ffd)
    assert np.array_equal(got["layouts"]["routepack"], oa["best_layout"])
    for key, qq, gg, x in (("baseline", q_id, g_id, x_ffd), ("reorder", q, g, x_ffd),
                           ("routepack", q, g, oa["best_layout"])):
        st, _, _, d = O.score(pb, w.lengths, qq, R, x, rank_load=gg, want_diag=True)
        assert st == 0
        want = bench._diag(d)
        for k in bench.DIAG_KEYS:
            assert got[key][k] == pytest.approx(want[k], rel=1e-6), (key, k)
    # LPT never leaves the rank loads more uneven than the identity does here
    assert got["reorder"]["cv_global"] <= got["baseline"]["cv_global"]
    # annealing starts from seeds that include FFD's layout and keeps the best
    assert got["routepack"]["joint"] <= got["reorder"]["joint"] + 1e-12


@gpu
@pytest.mark.parametrize("seed", range(6))
def test_project_demand_matches_oracle(seed):
    import oracle as O
    import paper_2608_12146_amd as rp
    rng = np.random.default_rng([23, seed])
    P = int(rng.choice([1, 2, 4, 8]))
    E = P * int(rng.integers(1, 9))
    L = int(rng.integers(1, 5))
    w = synth.make_tiny_random(400 + seed, n=int(rng.integers(1, 200)), layers=L, experts=E, top_k=min(2, E),
                               ranks=P, dp=1, cap=256)
    prob = rp.Problem.from_dict(synth.window_problem(w))
    agg = O.aggregate(w.demand)
    slot = np.stack([rng.permutation(E) for _ in range(L)]).astype(np.int32)
    _log(f"project_demand seed {seed}: N={w.n} L={L} E={E} P={P}")
    g, q = rp.project_demand(prob, agg, slot, w.demand)
    assert np.array_equal(g.cpu().numpy(), O.placement_load(agg, slot, P))
    assert np.array_equal(q.cpu().numpy(), O.project(w.demand, slot, P))
    g2, q2 = rp.project_demand(prob, agg, slot)
    assert q2 is None and np.array_equal(g2.cpu().numpy(), g.cpu().numpy())
    import torch
    big = torch.zeros(w.demand.size + 1, dtype=torch.int32, device="cuda")
    big[1:] = torch.as_tensor(w.demand.reshape(-1), device="cuda")
    off = big[1:].view(w.demand.shape)                    # rows not 16-byte aligned
    _, q3 = rp.project_demand(prob, agg, slot, off)
    assert np.array_equal(q3.cpu().numpy(), q.cpu().numpy())


@gpu
def test_project_demand_rejects_what_is_not_a_permutation():
    import paper_2608_12146_amd as rp
    w = synth.make_tiny_random(450, n=16, layers=2, experts=8, top_k=2, ranks=4, dp=1, cap=256)
    prob = rp.Problem.from_dict(synth.window_problem(w))
    agg = np.ones((2, 8), dtype=np.int64)
    good = np.tile(np.arange(8, dtype=np.int32), (2, 1))
    for bad in (8, -1):                                   # a slot out of range
        s = good.copy()
        s[1, 3] = bad
        with pytest.raises(rp.RoutepackError) as ei:
            rp.project_demand(prob, agg, s, w.demand)
        assert ei.value.code == -1
    s = good.copy()
    s[0, 5] = 2                                           # a slot taken twice
    with pytest.raises(rp.RoutepackError) as ei:
        rp.project_demand(prob, agg, s, w.demand)
    assert ei.value.code == -1
    g, _ = rp.project_demand(prob, agg, good)
    assert g.cpu().numpy().tolist() == [[2, 2, 2, 2]] * 2
