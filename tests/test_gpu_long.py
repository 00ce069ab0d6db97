"""Full-schedule annealing parity: every level's trace, the parents of every
resampling, the final population and x* equal the oracle's (on the
whole-schedule kernel where the window fits it).

- small (1024 samples, 16 layers, 64 experts, 8 ranks, 4 slots; population
  256, 1000 levels of 256 proposals, about 0.7 M evaluated moves), one and
  two attention stages: seconds;
- mid (4096 samples, 24 layers, 256 experts, 16 ranks, 8 slots; population
  1024, 2000 levels, about 43.5 M evaluated moves) with one EDP shard and one
  stage, two EDP shards, and two stages: about a minute and a quarter of
  oracle time each on 16 host threads;
- the first 1000 levels of heavy and the first 4 of stress: minutes of
  oracle time, so they run only when ROUTEPACK_LONG_TESTS=1."""
import os

import numpy as np
import pytest

import synth

gpu = pytest.mark.gpu
LONG = os.environ.get("ROUTEPACK_LONG_TESTS") == "1"


def _full_schedule(name, S, G=1, chunk=250, kernel="chain_run", levels=None):
    import oracle as O
    import paper_2608_12146_amd as rp
    from synth import windows as W
    w = synth.make_window(name, edp=G)
    pd = synth.window_problem(w, stages=S)
    pb = O.Problem.from_dict(pd)
    slot, _ = O.place(O.aggregate(w.demand), w.n_ranks)
    q = O.project(w.demand, slot, w.n_ranks)
    pr = O.pack_rows(pb, w.lengths, q, w.seed_pack, W.N_TRIALS, W.CHOICE_WIDTH, w.pop)
    assert pr["rc"] == 0
    all_temps = synth.anneal_temperatures(w.levels)
    n = levels or w.levels  # the first n levels of the window's schedule
    temps, t_after = all_temps[:n], (all_temps[n] if n < w.levels else 0.0)
    print(f"[gpu-long] {name} G={G} S={S}: {n} levels on the GPU", flush=True)
    g = rp.anneal(rp.Problem.from_dict(pd), w.lengths, q, pr["r_star"], pr["population"], temps,
                  W.STEPS_PER_LEVEL, w.seed_anneal, t_next=t_after)
    print(f"[gpu-long] {name} G={G} S={S}: level kernel {g['level_kernel']}", flush=True)
    if kernel:
        assert g["level_kernel"] == kernel
    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    gt, gp = g["trace"].cpu().numpy(), g["parents"].cpu().numpy()
    # The oracle in chunks of levels, each resuming from the last one's
    # population and x* (a resumed run equals an uninterrupted one), so that
    # every chunk is checked and reported as it ends.
    pop, bl, bs, evals = pr["population"], None, None, 0
    for lo in range(0, n, chunk):
        hi = min(n, lo + chunk)
        o = O.anneal(pb, w.lengths, q, pr["r_star"], pop, temps[lo:hi], W.STEPS_PER_LEVEL, w.seed_anneal,
                     t_next=temps[hi] if hi < n else t_after, sweep_offset=lo, best_layout=bl, best_score=bs,
                     n_threads=threads)
        assert o["rc"] == 0
        assert np.array_equal(gt[lo:hi], o["trace"]), (lo, hi)
        assert np.array_equal(gp[lo:hi], o["parents"]), (lo, hi)
        pop, bl, bs = o["population"], o["best_layout"], o["best_score"]
        evals += int(o["trace"][:, :, 7].sum())
        print(f"[gpu-long] {name} G={G} S={S}: levels {lo}-{hi - 1} equal on {threads} threads", flush=True)
    assert np.array_equal(g["population"].cpu().numpy(), pop)
    assert np.array_equal(g["best_layout"].cpu().numpy(), bl)
    assert np.array_equal(g["best_score"].cpu().numpy(), bs)
    print(f"[gpu-long] {name} G={G} S={S}: {evals} evaluated moves equal", flush=True)


@gpu
@pytest.mark.parametrize("S", [1, 2])
def test_anneal_full_schedule_small(S):
    _full_schedule("small", S)


@gpu
@pytest.mark.skipif(not LONG, reason="minutes of oracle time: set ROUTEPACK_LONG_TESTS=1")
@pytest.mark.parametrize("name", ["heavy", "stress"])
def test_anneal_full_schedule_large(name):
    """The first 1000 of the heavy-tail window's 2000 levels (population
    2048; about eleven minutes of oracle time, reported every 50 levels) and
    the first 4 of the stress window's 500 (population 4096; about two and a
    half minutes of oracle time per level, reported every level), on
    whichever level kernel the library picks (the per-level chain kernel:
    the cell array and lengths in HBM for the heavy-tail window, the 64-rank
    layout for the stress window)."""
    if name == "heavy":
        _full_schedule(name, 1, chunk=50, kernel=None, levels=1000)
    else:
        _full_schedule(name, 1, chunk=1, kernel=None, levels=4)


@gpu
@pytest.mark.parametrize("G,S", [(1, 1), (2, 1), (1, 2)])
def test_anneal_full_schedule_mid(G, S):
    """The common shape, two EDP shards (100 row-shards: two per lane) and
    two attention stages."""
    _full_schedule("mid", S, G)
