"""Parity on the heavy-tail (8192 samples, 48 layers, 256 experts, 32 ranks,
16 slots, cap 131072) and stress (32768 samples, 64 layers, 512 experts,
64 ranks, 32 slots, cap 131072, 4 GiB of demand) windows at full size.

Aggregation, placement, projection, packing and QualityDiversitySelect are
compared in full.
Annealing runs the full population for one level on the GPU; a sample of
members is recomputed by the oracle under their own replica ids (every
member's level is an independent chain given its start state)."""
import functools

import numpy as np
import pytest

import synth

gpu = pytest.mark.gpu


def _log(msg):
    print(f"[gpu-large] {msg}", flush=True)


@functools.lru_cache(maxsize=None)
def _prepared(name):
    import oracle as O
    w = synth.make_window(name)
    pd = synth.window_problem(w)
    pb = O.Problem.from_dict(pd)
    agg = O.aggregate(w.demand)
    slot, load = O.place(agg, w.n_ranks)
    q = O.project(w.demand, slot, w.n_ranks)
    pr = O.pack_rows(pb, w.lengths, q, w.seed_pack, synth.windows.N_TRIALS,
                     synth.windows.CHOICE_WIDTH, w.pop)
    assert pr["rc"] == 0
    return w, pd, pb, agg, slot, load, q, pr


@gpu
@pytest.mark.parametrize("name", ["heavy", "stress"])
def test_large_window_full_path(name):
    import oracle as O
    import paper_2608_12146_amd as rp
    _log(f"{name}: generating and running the oracle")
    w, pd, pb, agg, slot, load, q, pr = _prepared(name)
    prob = rp.Problem.from_dict(pd)
    _log(f"{name}: aggregate / place / project")
    g_agg = rp.aggregate_demand(prob, w.demand)
    assert np.array_equal(g_agg.cpu().numpy(), agg)
    g_slot, g_load, g_q = rp.place_experts(prob, g_agg, w.demand)
    assert np.array_equal(g_slot.cpu().numpy(), slot)
    assert np.array_equal(g_load.cpu().numpy(), load)
    assert np.array_equal(g_q.cpu().numpy(), q)
    _log(f"{name}: pack_rows")
    g = rp.pack_rows(prob, w.lengths, g_q, w.seed_pack, synth.windows.N_TRIALS,
                     synth.windows.CHOICE_WIDTH, w.pop)
    assert (g["r_star"], g["certified"], g["n_distinct"]) == (pr["r_star"], pr["certified"], pr["n_distinct"])
    assert np.array_equal(g["population"].cpu().numpy(), pr["population"])
    assert np.array_equal(g["scores"].cpu().numpy(), pr["scores"])
    _log(f"{name}: anneal one level, full population")
    temps = synth.anneal_temperatures(w.levels)
    K = synth.windows.STEPS_PER_LEVEL
    ga = rp.anneal(prob, w.lengths, g_q, pr["r_star"], g["population"], temps[:1], K, w.seed_anneal)
    ids = np.array([0, 1, 2, w.pop // 2, w.pop - 1], dtype=np.int32)
    _log(f"{name}: oracle on members {ids.tolist()}")
    oa = O.anneal(pb, w.lengths, q, pr["r_star"], pr["population"][ids], temps[:1], K, w.seed_anneal,
                  replica_ids=ids)
    assert oa["rc"] == 0
    gt = ga["trace"].cpu().numpy()[0]
    assert np.array_equal(gt[ids], oa["trace"][0])
    assert np.array_equal(ga["population"].cpu().numpy()[ids], oa["population"])


@gpu
@pytest.mark.parametrize("name", ["heavy", "stress"])
def test_large_window_select_population(name):
    """QualityDiversitySelect over the window's distinct seeds at full size:
    the order and the filled population equal the oracle's."""
    from oracle import qds
    import paper_2608_12146_amd as rp
    w, pd, pb, agg, slot, load, q, pr = _prepared(name)
    M = pr["n_distinct"]
    cands, s0 = pr["population"][:M], pr["scores"][:M, 0]
    _log(f"{name}: select_population over {M} candidates")
    want = qds.select(pb, w.lengths, q, pr["r_star"], cands, s0, w.seed_pack)
    got = rp.select_population(rp.Problem.from_dict(pd), w.lengths, q, pr["r_star"], cands, s0, w.seed_pack,
                               pop_size=w.pop)
    assert got["order"].cpu().tolist() == want.tolist()
    assert np.array_equal(got["population"].cpu().numpy(), qds.population(cands, want, w.pop))
