"""Parity on the heavy-tail (8192 samples, 48 layers, 256 experts, 32 ranks,
16 slots, cap 131072) and stress (32768 samples, 64 layers, 512 experts,
64 ranks, 32 slots, cap 131072, 4 GiB of demand) windows at full size.

Aggregation, placement, projection, packing and QualityDiversitySelect are
compared in full.
Annealing runs the full population over the schedule's first two levels
(each followed by systematic resampling) and one late level on the GPU; a
sample of members is recomputed by the oracle under their own replica ids
(every member's level is an independent chain given its start state), and
the parents of each resampling are checked for the whole population."""
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
    _anneal_two_levels_and_a_late_one(name, w, pb, q, pr, prob, g_q)


def _anneal_two_levels_and_a_late_one(name, w, pb, q, pr, prob, g_q):
    """Levels 0 and 1 of the window's schedule on the full population (two
    calls, the second resuming the first), then one late level resumed from
    the result.  The oracle recomputes sampled members under their replica
    ids (a member's level is an independent chain given its start state);
    every resampling's parents are checked for the whole population against
    the oracle's systematic resampling of the GPU's terminal energies."""
    import oracle as O
    import paper_2608_12146_amd as rp
    temps = synth.anneal_temperatures(w.levels)
    K = synth.windows.STEPS_PER_LEVEL
    late = w.levels * 3 // 4
    ids = np.array([0, 1, 2, w.pop // 3, w.pop // 2, w.pop - 1], dtype=np.int32)
    pop0 = pr["population"]
    _log(f"{name}: level 0, full population ({w.pop} members)")
    a = rp.anneal(prob, w.lengths, g_q, pr["r_star"], pop0, temps[:1], K, w.seed_anneal, t_next=temps[1])
    ta, pa = a["trace"].cpu().numpy()[0], a["parents"].cpu().numpy()[0]
    popa = a["population"].cpu().numpy()
    _log(f"{name}: level 0 on the oracle for members {ids.tolist()} ({a['level_kernel']} kernel)")
    oa = O.anneal(pb, w.lengths, q, pr["r_star"], pop0[ids], temps[:1], K, w.seed_anneal, replica_ids=ids)
    assert oa["rc"] == 0
    assert np.array_equal(ta[ids], oa["trace"][0])
    # resampling of the whole population from the GPU's terminal energies
    en = O.energy(pb, ta[:, 0:3])
    assert np.array_equal(pa, O.resample(en, temps[0], temps[1], w.seed_anneal, 0))
    # children of the recomputed members carry their terminal states
    term = dict(zip(ids.tolist(), oa["population"]))
    kids = [m for m in range(w.pop) if int(pa[m]) in term]
    assert kids
    for m in kids:
        assert np.array_equal(popa[m], term[int(pa[m])]), m
    # x*: the lexicographic min of the start population and every member's best
    best = min([tuple(x) for x in pr["scores"]] + [tuple(x) for x in ta[:, 3:6]])
    assert tuple(a["best_score"].cpu().numpy()) == best

    _log(f"{name}: level 1 resumed, full population")
    b = rp.anneal(prob, w.lengths, g_q, pr["r_star"], a["population"], temps[1:2], K, w.seed_anneal,
                  t_next=temps[2], sweep_offset=1, best_layout=a["best_layout"], best_score=a["best_score"])
    tb, pbp = b["trace"].cpu().numpy()[0], b["parents"].cpu().numpy()[0]
    kid_ids = np.array(kids[:6], dtype=np.int32)
    ob = O.anneal(pb, w.lengths, q, pr["r_star"], popa[kid_ids], temps[1:2], K, w.seed_anneal,
                  sweep_offset=1, replica_ids=kid_ids)
    assert ob["rc"] == 0
    assert np.array_equal(tb[kid_ids], ob["trace"][0])
    en = O.energy(pb, tb[:, 0:3])
    assert np.array_equal(pbp, O.resample(en, temps[1], temps[2], w.seed_anneal, 1))

    _log(f"{name}: level {late} resumed from that population")
    popb = b["population"].cpu().numpy()
    c = rp.anneal(prob, w.lengths, g_q, pr["r_star"], b["population"], temps[late:late + 1], K,
                  w.seed_anneal, sweep_offset=late, best_layout=b["best_layout"], best_score=b["best_score"])
    tc = c["trace"].cpu().numpy()[0]
    oc = O.anneal(pb, w.lengths, q, pr["r_star"], popb[ids], temps[late:late + 1], K, w.seed_anneal,
                  sweep_offset=late, replica_ids=ids)
    assert oc["rc"] == 0
    assert np.array_equal(tc[ids], oc["trace"][0])
    assert np.array_equal(c["population"].cpu().numpy()[ids], oc["population"])
    assert (c["parents"].cpu().numpy() == -1).all()
    _log(f"{name}: {int(ta[:, 7].sum() + tb[:, 7].sum() + tc[:, 7].sum())} evaluated moves on the GPU")


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
