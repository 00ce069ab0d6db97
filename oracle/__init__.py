"""CPU oracle for the RoutePack planner hot path -- TEST INFRASTRUCTURE ONLY.

Only tests/, the smoke check and the CPU-baseline leg of the benchmark may
import this package.  It wraps the plain C oracle (routepack_oracle.c) with
ctypes; it shares nothing with the HIP library.  Every function follows the
passage of arXiv 2608.12146 named in its docstring.

Parity-unpinned parts (see the C file header): the full annealing trajectory.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "routepack_oracle.c")
_LIB_PATH = os.path.join(_HERE, "librp_oracle.so")
_lib = None
_lock = threading.Lock()

OK, INVALID, INFEASIBLE, HEURISTIC, LAYOUT, OVERFLOW, INTERNAL = 0, -1, -2, -3, -4, -5, -7


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no contraction, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-ffp-contract=off", "-fno-fast-math",
                               "-Wall", "-pthread", "-shared", "-fPIC", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class _Problem(C.Structure):
    _fields_ = [("n_samples", C.c_int32), ("n_layers", C.c_int32), ("n_experts", C.c_int32),
                ("top_k", C.c_int32), ("n_ranks", C.c_int32), ("n_dp", C.c_int32),
                ("n_edp", C.c_int32), ("dp_to_edp", C.POINTER(C.c_int32)),
                ("capacity", C.c_int64), ("n_stages", C.c_int32),
                ("alpha_fp", C.POINTER(C.c_int64)), ("beta_fp", C.POINTER(C.c_int64)),
                ("frac_bits", C.c_int32), ("min_rows", C.c_int32)]


class _AnnealParams(C.Structure):
    _fields_ = [("n_sweeps", C.c_int32), ("steps_per_sweep", C.c_int32),
                ("temperatures", C.POINTER(C.c_double)), ("t_next", C.c_double),
                ("p_guide_u32", C.c_uint32), ("rho_u32", C.c_uint32), ("seed", C.c_uint64),
                ("sweep_offset", C.c_int32), ("init_incumbent", C.c_int32)]


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
                build(force=True)
            lib = C.CDLL(_LIB_PATH)
            lib.or_exp_det.restype = C.c_double
            lib.or_exp_det.argtypes = [C.c_double]
            _lib = lib
    return _lib


def _p(a, ctype):
    return a.ctypes.data_as(C.POINTER(ctype))


class Problem:
    """Problem description (Sec. 3.1-3.4): sizes, topology {D_g}, capacity C,
    stage coefficients alpha_s, beta_s at 2^frac_bits, pipeline row bound."""

    def __init__(self, n_samples, n_layers, n_experts, top_k, n_ranks, n_dp, n_edp, dp_to_edp,
                 capacity, alpha_fp, beta_fp, frac_bits=12, min_rows=1):
        self.dp_to_edp = np.ascontiguousarray(dp_to_edp, dtype=np.int32)
        self.alpha_fp = np.ascontiguousarray(alpha_fp, dtype=np.int64)
        self.beta_fp = np.ascontiguousarray(beta_fp, dtype=np.int64)
        assert self.alpha_fp.shape == self.beta_fp.shape
        self.n_samples, self.n_layers, self.n_experts = int(n_samples), int(n_layers), int(n_experts)
        self.top_k, self.n_ranks, self.n_dp, self.n_edp = int(top_k), int(n_ranks), int(n_dp), int(n_edp)
        self.capacity, self.frac_bits, self.min_rows = int(capacity), int(frac_bits), int(min_rows)
        self._c = _Problem(self.n_samples, self.n_layers, self.n_experts, self.top_k, self.n_ranks,
                           self.n_dp, self.n_edp, _p(self.dp_to_edp, C.c_int32), self.capacity,
                           len(self.alpha_fp), _p(self.alpha_fp, C.c_int64),
                           _p(self.beta_fp, C.c_int64), self.frac_bits, self.min_rows)

    @classmethod
    def from_dict(cls, d):
        return cls(**d)

    @property
    def ref(self):
        return C.byref(self._c)


def philox4x64(counter, key):
    """One Philox4x64-10 block (Salmon et al., SC'11) for a 4-word counter and
    2-word key; returns 4 uint64."""
    lib = _load()
    c = np.ascontiguousarray(counter, dtype=np.uint64)
    k = np.ascontiguousarray(key, dtype=np.uint64)
    out = np.zeros(4, dtype=np.uint64)
    lib.or_philox4x64(_p(c, C.c_uint64), _p(k, C.c_uint64), _p(out, C.c_uint64))
    return out


def exp_det(x):
    """Deterministic exp(x) for x <= 0 (Cody-Waite reduction, Taylor degree 13)."""
    lib = _load()
    xs = np.atleast_1d(np.asarray(x, dtype=np.float64))
    return np.array([lib.or_exp_det(float(v)) for v in xs])


def aggregate(demand):
    """L_{l,e} = sum_i a_{i,l,e} (Sec. 3.3), int64 [L][E]."""
    lib = _load()
    d = np.ascontiguousarray(demand, dtype=np.int32)
    N, L, E = d.shape
    out = np.zeros((L, E), dtype=np.int64)
    lib.or_aggregate(C.c_int32(N), C.c_int32(L), C.c_int32(E), _p(d, C.c_int32), _p(out, C.c_int64))
    return out


def place(agg, n_ranks):
    """Layer-local LPT (Alg. 1): returns (slot_of [L][E] = pi_l(e), rank_load [L][P])."""
    lib = _load()
    a = np.ascontiguousarray(agg, dtype=np.int64)
    L, E = a.shape
    slot = np.zeros((L, E), dtype=np.int32)
    load = np.zeros((L, n_ranks), dtype=np.int64)
    rc = lib.or_place(C.c_int32(L), C.c_int32(E), C.c_int32(n_ranks), _p(a, C.c_int64),
                      _p(slot, C.c_int32), _p(load, C.c_int64))
    if rc:
        raise ValueError(f"or_place rc={rc}")
    return slot, load


def project(demand, slot_of, n_ranks):
    """q_{i,l,p} = sum_{e: owner(pi_l(e)) = p} a_{i,l,e} (Eq. physical-rank-demand)."""
    lib = _load()
    d = np.ascontiguousarray(demand, dtype=np.int32)
    s = np.ascontiguousarray(slot_of, dtype=np.int32)
    N, L, E = d.shape
    q = np.zeros((N, L, n_ranks), dtype=np.int32)
    rc = lib.or_project(C.c_int32(N), C.c_int32(L), C.c_int32(E), C.c_int32(n_ranks),
                        _p(d, C.c_int32), _p(s, C.c_int32), _p(q, C.c_int32))
    if rc:
        raise ValueError(f"or_project rc={rc}")
    return q


def placement_load(agg, slot_of, n_ranks):
    """G_{l,p} = sum of agg[l][e] over the experts e with owner(pi_l(e)) = p,
    owner(v) = v // H, H = E / P (Eq. placement-load), for any placement."""
    a = np.asarray(agg, dtype=np.int64)
    s = np.asarray(slot_of, dtype=np.int64)
    L, E = a.shape
    H = E // n_ranks
    G = np.zeros((L, n_ranks), dtype=np.int64)
    for l in range(L):
        for e in range(E):
            G[l, s[l, e] // H] += a[l, e]
    return G


def score(prob: Problem, lengths, q, n_rows, layout, rank_load=None, want_J=False, want_diag=False):
    """Exact fixed-point score of one layout (Eqs. 11-15) -> (status, s[3], J, diag)."""
    lib = _load()
    t = np.ascontiguousarray(lengths, dtype=np.int32)
    qq = np.ascontiguousarray(q, dtype=np.int32)
    lay = np.ascontiguousarray(layout, dtype=np.int32)
    s = np.zeros(3, dtype=np.int64)
    J = np.zeros(n_rows * prob.n_edp, dtype=np.int64) if want_J else None
    diag = np.zeros(8, dtype=np.float64) if want_diag else None
    rl = None if rank_load is None else np.ascontiguousarray(rank_load, dtype=np.int64)
    st = lib.or_score(prob.ref, _p(t, C.c_int32), _p(qq, C.c_int32), C.c_int32(n_rows),
                      _p(lay, C.c_int32), _p(s, C.c_int64),
                      _p(J, C.c_int64) if J is not None else None,
                      _p(diag, C.c_double) if diag is not None else None,
                      _p(rl, C.c_int64) if rl is not None else None)
    return st, s, J, diag


def pack_rows(prob: Problem, lengths, q, seed, n_trials, width, pop):
    """Row-count search + FixedRowFFD + Alg. 2 seeding.
    Returns dict(rc, r_star, certified, population [pop][N], scores [pop][3],
    r_lb, n_distinct, n_trials_ok)."""
    lib = _load()
    t = np.ascontiguousarray(lengths, dtype=np.int32)
    qq = np.ascontiguousarray(q, dtype=np.int32)
    N = prob.n_samples
    popl = np.zeros((pop, N), dtype=np.int32)
    sc = np.zeros((pop, 3), dtype=np.int64)
    r_star = C.c_int32(0)
    cert = C.c_int32(0)
    extra = np.zeros(3, dtype=np.int32)
    rc = lib.or_pack_rows(prob.ref, _p(t, C.c_int32), _p(qq, C.c_int32), C.c_uint64(seed),
                          C.c_int32(n_trials), C.c_int32(width), C.c_int32(pop),
                          C.byref(r_star), C.byref(cert), _p(popl, C.c_int32), _p(sc, C.c_int64),
                          _p(extra, C.c_int32))
    return dict(rc=rc, r_star=r_star.value, certified=bool(cert.value), population=popl,
                scores=sc, r_lb=int(extra[0]), n_distinct=int(extra[1]), n_trials_ok=int(extra[2]))


def seed_trial(prob: Problem, lengths, q, n_rows, width, seed, trial):
    """One randomized seed trial of Alg. 2 with its steps exposed (Sec. 4.1.1):
    dict(ok, pi = the WindowShuffle order, cellk = the RandomizedBestFit cell
    k in [0, R*D) of each sample, layout = the cell id r*D + d after
    EDPAwarePair)."""
    lib = _load()
    t = np.ascontiguousarray(lengths, dtype=np.int32)
    qq = np.ascontiguousarray(q, dtype=np.int32)
    N = prob.n_samples
    pi = np.full(N, -1, dtype=np.int32)
    ck = np.full(N, -1, dtype=np.int32)
    lay = np.full(N, -1, dtype=np.int32)
    rc = lib.or_seed_trial(prob.ref, _p(t, C.c_int32), _p(qq, C.c_int32), C.c_int32(n_rows),
                           C.c_int32(width), C.c_uint64(seed), C.c_uint64(trial),
                           _p(pi, C.c_int32), _p(ck, C.c_int32), _p(lay, C.c_int32))
    if rc < 0:
        raise ValueError(f"or_seed_trial rc={rc}")
    return dict(ok=bool(rc), pi=pi, cellk=ck, layout=lay)


def edp_pair(prob: Problem, q, n_rows, cellk, width, seed, trial):
    """EDPAwarePair alone (Sec. 4.1.1) on completed cells cellk[i] in
    [0, R*D): returns the layout (cell id r*D + d per sample)."""
    lib = _load()
    qq = np.ascontiguousarray(q, dtype=np.int32)
    ck = np.ascontiguousarray(cellk, dtype=np.int32)
    lay = np.full(prob.n_samples, -1, dtype=np.int32)
    rc = lib.or_edp_pair(prob.ref, _p(qq, C.c_int32), C.c_int32(n_rows), _p(ck, C.c_int32),
                         C.c_int32(width), C.c_uint64(seed), C.c_uint64(trial), _p(lay, C.c_int32))
    if rc:
        raise ValueError(f"or_edp_pair rc={rc}")
    return lay


def energy(prob: Problem, scores):
    """Eq. pa-energy of score triples [n][3]: (S0 + 1e-6 S1) + 1e-9 S2 with
    S_i = s_i / (2^F C)."""
    lib = _load()
    s = np.ascontiguousarray(np.asarray(scores, dtype=np.int64).reshape(-1, 3))
    out = np.zeros(len(s), dtype=np.float64)
    lib.or_energy(C.c_int32(len(s)), _p(s, C.c_int64), C.c_int32(prob.frac_bits),
                  C.c_int64(prob.capacity), _p(out, C.c_double))
    return out


def resample(energies, t_cur, t_next, seed, level):
    """Systematic resampling of one level boundary -> parent indices [pop]."""
    lib = _load()
    e = np.ascontiguousarray(energies, dtype=np.float64)
    par = np.zeros(len(e), dtype=np.int32)
    lib.or_resample(C.c_int32(len(e)), _p(e, C.c_double), C.c_double(t_cur), C.c_double(t_next),
                    C.c_uint64(seed), C.c_int32(level), _p(par, C.c_int32))
    return par


def resample_at(energies, t_cur, t_next, V):
    """The systematic resampling step for a given uniform V in [0, 2^32)
    (u_0 = V / (2^32 P)) -> parent indices [pop]."""
    lib = _load()
    e = np.ascontiguousarray(energies, dtype=np.float64)
    par = np.zeros(len(e), dtype=np.int32)
    lib.or_resample_at(C.c_int32(len(e)), _p(e, C.c_double), C.c_double(t_cur), C.c_double(t_next),
                       C.c_uint64(V), _p(par, C.c_int32))
    return par


def anneal(prob: Problem, lengths, q, n_rows, population, temperatures, steps_per_sweep, seed,
           t_next=0.0, sweep_offset=0, p_guide_u32=0xCCCCCCCD, rho_u32=0x40000000,
           best_layout=None, best_score=None, want_trace=True, want_parents=True,
           want_steps=False, n_threads=None, check_full=False, replica_ids=None):
    """Population annealing (Alg. 3) over len(temperatures) levels.
    Returns dict(rc, population, best_layout, best_score, trace, parents, steps)."""
    lib = _load()
    t = np.ascontiguousarray(lengths, dtype=np.int32)
    qq = np.ascontiguousarray(q, dtype=np.int32)
    popl = np.array(population, dtype=np.int32, copy=True, order="C")
    P, N = popl.shape
    temps = np.ascontiguousarray(temperatures, dtype=np.float64)
    ns = len(temps)
    init = best_layout is None
    bl = np.zeros(N, dtype=np.int32) if init else np.array(best_layout, dtype=np.int32, copy=True)
    bs = np.zeros(3, dtype=np.int64) if init else np.array(best_score, dtype=np.int64, copy=True)
    trace = np.zeros((ns, P, 8), dtype=np.int64) if want_trace else None
    parents = np.zeros((ns, P), dtype=np.int32) if want_parents else None
    steps = np.zeros((ns, P, steps_per_sweep), dtype=np.uint8) if want_steps else None
    ap = _AnnealParams(ns, steps_per_sweep, _p(temps, C.c_double), float(t_next), p_guide_u32,
                       rho_u32, seed, sweep_offset, 1 if init else 0)
    if n_threads is None:
        n_threads = min(P, os.cpu_count() or 1, 16)
    rid = None if replica_ids is None else np.ascontiguousarray(replica_ids, dtype=np.int32)
    assert rid is None or rid.shape == (P,)
    rc = lib.or_anneal(prob.ref, _p(t, C.c_int32), _p(qq, C.c_int32), C.c_int32(n_rows),
                       C.c_int32(P), _p(popl, C.c_int32), C.byref(ap), _p(bl, C.c_int32),
                       _p(bs, C.c_int64),
                       _p(trace, C.c_int64) if trace is not None else None,
                       _p(parents, C.c_int32) if parents is not None else None,
                       _p(steps, C.c_uint8) if steps is not None else None,
                       C.c_int32(n_threads), C.c_int32(1 if check_full else 0),
                       _p(rid, C.c_int32) if rid is not None else None)
    return dict(rc=rc, population=popl, best_layout=bl, best_score=bs, trace=trace,
                parents=parents, steps=steps, n_threads=n_threads)
