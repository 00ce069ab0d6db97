"""Window recipes and the seeded generator.

Every window is one optimizer step: N samples with lengths t_i and replayed
routing counts a[i, l, e] (the routing-replay input of the paper's
problem statement, Sec. 2.1, Eq. routing-replay-input).  Counts are drawn as a
multinomial of k * t_i assignments over a per-layer Zipf profile and then
capped at t_i (a top-k router sends a token to k *distinct* experts, so no
expert can receive more than t_i assignments from one sample); the excess is
re-drawn over the experts still below the cap until none exceeds it.

Named windows (sizes are the contract; the seed fixes the values):

  tiny   64 samples, t ~ U{16..512}; 4 layers, 16 experts, top-2, Zipf 1.0
         over a seeded per-layer permutation; 4 EP ranks, 2 DP slots,
         cap 1024; population 8, 200 levels.
  small  1024 samples, t ~ lognormal(median 2048, sigma 0.8) clipped
         [64, 16384]; 16 layers, 64 experts, top-6, Zipf 1.1 with per-sample
         Dirichlet(50 p) perturbation; 8 ranks, 4 slots, cap 32768;
         population 256, 1000 levels.
  mid    4096 samples, lognormal(4096, 1.0) clipped [128, 32768]; 24 layers,
         256 experts, top-8, Zipf 1.2, permutation drifting 10% per layer;
         16 ranks, 8 slots, cap 65536; population 1024, 2000 levels.
  heavy  8192 samples, 80% lognormal(2048, 1.0) clipped [64, 65536] + 20%
         U{32768..65536}; 48 layers, 256 experts, top-8, Zipf 1.3 with 5 hot
         experts per layer at 4x weight; 32 ranks, 16 slots, cap 131072;
         population 2048, 2000 levels.
  stress 32768 samples, lognormal(4096, 1.2) clipped [64, 65536]; 64 layers,
         512 experts, top-8, Zipf 1.1 drifting 10% per layer; 64 ranks,
         32 slots, cap 131072; population 4096, 500 levels.
"""
from __future__ import annotations

import dataclasses
import os
from typing import Optional

import numpy as np

WINDOWS = {
    "tiny": dict(index=0, n=64, lengths=("uniform", 16, 512), layers=4,
                 experts=16, top_k=2, zipf=1.0, mode="perm", ranks=4, dp=2,
                 cap=1024, pop=8, levels=200),
    "small": dict(index=1, n=1024, lengths=("lognormal", 2048, 0.8, 64, 16384),
                  layers=16, experts=64, top_k=6, zipf=1.1, mode="dirichlet",
                  ranks=8, dp=4, cap=32768, pop=256, levels=1000),
    "mid": dict(index=2, n=4096, lengths=("lognormal", 4096, 1.0, 128, 32768),
                layers=24, experts=256, top_k=8, zipf=1.2, mode="drift",
                ranks=16, dp=8, cap=65536, pop=1024, levels=2000),
    "heavy": dict(index=3, n=8192, lengths=("heavy", 2048, 1.0, 64, 65536,
                                            0.2, 32768, 65536),
                  layers=48, experts=256, top_k=8, zipf=1.3, mode="hot",
                  ranks=32, dp=16, cap=131072, pop=2048, levels=2000),
    "stress": dict(index=4, n=32768, lengths=("lognormal", 4096, 1.2, 64, 65536),
                   layers=64, experts=512, top_k=8, zipf=1.1, mode="drift",
                   ranks=64, dp=32, cap=131072, pop=4096, levels=500),
}

# Planner knobs shared by every window (fixed-point scale, attention
# coefficients in raw tokens: a = 1, b = 1/4096 -> alpha_fp = 4096, beta_fp = 1
# at 12 fractional bits; proposal budget per level; seeding budget).
FRAC_BITS = 12
ALPHA_FP = 4096
BETA_FP = 1
# Two attention stages (the KDA + MLA stack of Sec. 2.2): a linear stage
# (a = 1, b = 0) and one with a quadratic term (a = 1/2, b = 1/4096), at 12
# fractional bits.
ALPHA_FP_2 = (4096, 2048)
BETA_FP_2 = (0, 1)
STEPS_PER_LEVEL = 256
N_TRIALS = 16
CHOICE_WIDTH = 4
P_GUIDE_U32 = 0xCCCCCCCD   # 0.8 * 2^32, rounded up
RHO_U32 = 0x40000000       # 0.25 * 2^32
T_FIRST = 1e-3
T_LAST = 1e-6


@dataclasses.dataclass
class Window:
    name: str
    lengths: np.ndarray        # int32 [N]
    demand: np.ndarray         # int32 [N][L][E]
    top_k: int
    n_ranks: int
    n_dp: int
    capacity: int
    pop: int
    levels: int
    dp_to_edp: np.ndarray      # int32 [D]
    seed_pack: int
    seed_anneal: int

    @property
    def n(self): return int(self.demand.shape[0])
    @property
    def n_layers(self): return int(self.demand.shape[1])
    @property
    def n_experts(self): return int(self.demand.shape[2])
    @property
    def n_edp(self): return int(self.dp_to_edp.max()) + 1 if len(self.dp_to_edp) else 0


def _lengths(rng, spec, n):
    kind = spec[0]
    if kind == "uniform":
        return rng.integers(spec[1], spec[2] + 1, size=n)
    if kind == "lognormal":
        _, med, sig, lo, hi = spec
        x = np.rint(np.exp(rng.normal(np.log(med), sig, size=n)))
        return np.clip(x, lo, hi)
    if kind == "heavy":
        _, med, sig, lo, hi, frac, ulo, uhi = spec
        x = np.clip(np.rint(np.exp(rng.normal(np.log(med), sig, size=n))), lo, hi)
        n_heavy = int(round(frac * n))
        pos = rng.choice(n, size=n_heavy, replace=False)
        x[pos] = rng.integers(ulo, uhi + 1, size=n_heavy)
        return x
    raise ValueError(kind)


def _drift(rng, perm, frac):
    """Cyclically rotate round(frac*E) randomly chosen positions of perm."""
    e = perm.shape[0]
    m = int(round(frac * e))
    if m < 2:
        return perm.copy()
    pos = np.sort(rng.choice(e, size=m, replace=False))
    out = perm.copy()
    out[pos] = perm[np.roll(pos, 1)]
    return out


def _capped_multinomial(rng, totals, p, cap):
    """Multinomial(totals, p) per row, then cap each count at cap[row] and
    re-draw the excess over the experts still below the cap."""
    counts = rng.multinomial(totals, p)
    capc = cap[:, None]
    for _ in range(64):
        over = counts > capc
        if not over.any():
            break
        excess = np.where(over, counts - capc, 0).sum(axis=1)
        counts = np.minimum(counts, capc)
        rows = np.nonzero(excess)[0]
        pr = (p[rows] if p.ndim == 2 else np.broadcast_to(p, (len(rows), p.shape[-1])))
        room = counts[rows] < capc[rows]
        q = np.where(room, pr, 0.0)
        q = q / q.sum(axis=1, keepdims=True)
        counts[rows] += rng.multinomial(excess[rows], q)
    else:
        raise RuntimeError("capping did not converge")
    assert (counts <= capc).all()
    return counts


def _layer_profiles(rng, cfg):
    """Per-layer Zipf profiles p_l over the experts (structural stream)."""
    L, E = cfg["layers"], cfg["experts"]
    s, mode = cfg["zipf"], cfg["mode"]
    profiles = np.empty((L, E), dtype=np.float64)
    perm = rng.permutation(E)
    for l in range(L):
        if mode in ("perm", "dirichlet", "hot"):
            perm = rng.permutation(E)
        elif mode == "drift" and l > 0:
            perm = _drift(rng, perm, 0.10)
        rank = np.empty(E, dtype=np.int64)
        rank[perm] = np.arange(E)
        p = (rank + 1.0) ** (-s)
        if mode == "hot":
            hot = rng.choice(E, size=5, replace=False)
            p[hot] *= 4.0
        profiles[l] = p / p.sum()
    return profiles


def _layer_demand(args):
    """Counts of one layer from its own stream: [2608, 12146, index, 1 + l]."""
    index, l, p, mode, k, t = args
    rng = np.random.default_rng([2608, 12146, index, 1 + l])
    if mode == "dirichlet":
        pp = rng.dirichlet(50.0 * p, size=t.shape[0])
        pp = np.maximum(pp, 0.0)
        pp = pp / pp.sum(axis=1, keepdims=True)
    else:
        pp = p
    return _capped_multinomial(rng, k * t, pp, t).astype(np.int32)


def _demand(rng, cfg, t, workers=None):
    n, L, E, k = cfg["n"], cfg["layers"], cfg["experts"], cfg["top_k"]
    profiles = _layer_profiles(rng, cfg)
    out = np.empty((n, L, E), dtype=np.int32)
    jobs = [(cfg["index"], l, profiles[l], cfg["mode"], k, t) for l in range(L)]
    if workers is None:
        workers = min(16, os.cpu_count() or 1) if n * L * E >= (1 << 22) else 1
    if workers > 1:
        import multiprocessing as mp
        with mp.get_context("fork").Pool(workers) as pool:
            for l, counts in enumerate(pool.imap(_layer_demand, jobs)):
                out[:, l, :] = counts
    else:
        for l, job in enumerate(jobs):
            out[:, l, :] = _layer_demand(job)
    return out


def _cache_dir():
    d = os.environ.get("ROUTEPACK_SYNTH_CACHE")
    if d is None:
        d = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                         "_build", "synth_cache")
    return d


def make_window(name: str, cache: bool = True, edp: Optional[int] = None) -> Window:
    """Draw (or load from the on-disk cache) the named window.

    edp: number of EDP shards G (contiguous slot blocks); default 1."""
    cfg = WINDOWS[name]
    c = cfg["index"]
    n = cfg["n"]
    path = os.path.join(_cache_dir(), f"{name}.npz")
    lengths = demand = None
    if cache and os.path.exists(path):
        with np.load(path, allow_pickle=False) as z:
            lengths, demand = z["lengths"], z["demand"]
    if lengths is None:
        rng = np.random.default_rng([2608, 12146, c])
        lengths = _lengths(rng, cfg["lengths"], n).astype(np.int32)
        demand = _demand(rng, cfg, lengths.astype(np.int64))
        if cache:
            os.makedirs(_cache_dir(), exist_ok=True)
            tmp = path + f".tmp{os.getpid()}.npz"
            np.savez(tmp, lengths=lengths, demand=demand)
            os.replace(tmp, path)
    g = 1 if edp is None else int(edp)
    D = cfg["dp"]
    assert D % g == 0
    dp_to_edp = (np.arange(D) // (D // g)).astype(np.int32)
    return Window(name=name, lengths=lengths, demand=demand, top_k=cfg["top_k"],
                  n_ranks=cfg["ranks"], n_dp=D, capacity=cfg["cap"], pop=cfg["pop"],
                  levels=cfg["levels"], dp_to_edp=dp_to_edp,
                  seed_pack=2000 + c, seed_anneal=1000 + c)


def make_tiny_random(seed: int, n: int = 8, layers: int = 2, experts: int = 4,
                     top_k: int = 2, ranks: int = 2, dp: int = 2, edp: int = 1,
                     cap: int = 64, tmin: int = 1, tmax: Optional[int] = None,
                     pop: int = 4, levels: int = 4) -> Window:
    """A small random instance for brute force and property tests."""
    rng = np.random.default_rng([7, seed])
    tmax = cap if tmax is None else tmax
    t = rng.integers(tmin, tmax + 1, size=n).astype(np.int64)
    demand = np.empty((n, layers, experts), dtype=np.int32)
    for l in range(layers):
        p = rng.dirichlet(np.ones(experts))
        demand[:, l, :] = _capped_multinomial(rng, top_k * t, p, t)
    dp_to_edp = (np.arange(dp) // (dp // edp)).astype(np.int32)
    return Window(name=f"rand{seed}", lengths=t.astype(np.int32), demand=demand,
                  top_k=top_k, n_ranks=ranks, n_dp=dp, capacity=cap, pop=pop,
                  levels=levels, dp_to_edp=dp_to_edp, seed_pack=seed, seed_anneal=seed + 1)


def anneal_temperatures(levels: int, t_first: float = T_FIRST, t_last: float = T_LAST):
    """Geometric schedule t_first * (t_last/t_first)^(n/(levels-1)), as float64."""
    if levels == 1:
        return np.array([t_first], dtype=np.float64)
    n = np.arange(levels, dtype=np.float64)
    return t_first * (t_last / t_first) ** (n / (levels - 1))


def window_problem(w: Window, stages: int = 1) -> dict:
    """The scalar problem description shared by both implementations; stages
    selects one attention stage or the two-stage (linear + quadratic) cost."""
    assert stages in (1, 2)
    alpha = [ALPHA_FP] if stages == 1 else list(ALPHA_FP_2)
    beta = [BETA_FP] if stages == 1 else list(BETA_FP_2)
    return dict(n_samples=w.n, n_layers=w.n_layers, n_experts=w.n_experts,
                top_k=w.top_k, n_ranks=w.n_ranks, n_dp=w.n_dp, n_edp=w.n_edp,
                dp_to_edp=w.dp_to_edp.astype(np.int32), capacity=int(w.capacity),
                alpha_fp=np.array(alpha, dtype=np.int64),
                beta_fp=np.array(beta, dtype=np.int64),
                frac_bits=FRAC_BITS, min_rows=1)
