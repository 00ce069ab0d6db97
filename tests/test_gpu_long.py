"""Full-schedule annealing parity on the default whole-schedule kernel:
every level's trace, the parents of every resampling, the final population
and x* equal the oracle's.

- small (1024 samples, 16 layers, 64 experts, 8 ranks, 4 slots; population
  256, 1000 levels of 256 proposals, about 0.7 M evaluated moves), one and
  two attention stages: seconds;
- mid (4096 samples, 24 layers, 256 experts, 16 ranks, 8 slots; population
  1024, 2000 levels, about 43.5 M evaluated moves) with one or two EDP
  shards or two stages: over a minute of oracle time each, so it runs only
  when ROUTEPACK_LONG_TESTS=1."""
import os

import numpy as np
import pytest

import synth

gpu = pytest.mark.gpu
LONG = os.environ.get("ROUTEPACK_LONG_TESTS") == "1"


def _full_schedule(name, S, G=1):
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
    temps = synth.anneal_temperatures(w.levels)
    print(f"[gpu-long] {name} G={G} S={S}: {w.levels} levels on the GPU", flush=True)
    g = rp.anneal(rp.Problem.from_dict(pd), w.lengths, q, pr["r_star"], pr["population"], temps,
                  W.STEPS_PER_LEVEL, w.seed_anneal)
    assert g["level_kernel"] == "chain_run"
    threads = min(16, os.cpu_count() or 1)
    print(f"[gpu-long] {name} G={G} S={S}: the oracle on {threads} threads", flush=True)
    o = O.anneal(pb, w.lengths, q, pr["r_star"], pr["population"], temps, W.STEPS_PER_LEVEL, w.seed_anneal,
                 n_threads=threads)
    assert o["rc"] == 0
    assert np.array_equal(g["trace"].cpu().numpy(), o["trace"])
    assert np.array_equal(g["parents"].cpu().numpy(), o["parents"])
    assert np.array_equal(g["population"].cpu().numpy(), o["population"])
    assert np.array_equal(g["best_layout"].cpu().numpy(), o["best_layout"])
    assert np.array_equal(g["best_score"].cpu().numpy(), o["best_score"])
    print(f"[gpu-long] {name} G={G} S={S}: {int(o['trace'][:, :, 7].sum())} evaluated moves equal", flush=True)


@gpu
@pytest.mark.parametrize("S", [1, 2])
def test_anneal_full_schedule_small(S):
    _full_schedule("small", S)


@gpu
@pytest.mark.skipif(not LONG, reason="minutes of oracle time: set ROUTEPACK_LONG_TESTS=1")
@pytest.mark.parametrize("G,S", [(1, 1), (2, 1), (1, 2)])
def test_anneal_full_schedule_mid(G, S):
    """The common shape, two EDP shards (100 row-shards: two per lane) and
    two attention stages."""
    _full_schedule("mid", S, G)
