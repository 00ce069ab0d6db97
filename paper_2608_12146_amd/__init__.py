"""MI355X (gfx950) RoutePack planner hot path -- Python binding.

A thin ctypes layer over the C-ABI in include/routepack.h (libroutepack.so).
It only marshals arguments: torch supplies device memory and the current HIP
stream, and every step of the path runs in the library's HIP kernels.  There
is no CPU fallback: importing works without a GPU, but every call raises if
the library or a GPU is missing.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libroutepack.so")

ERRORS = {0: "ok", -1: "invalid argument", -2: "infeasible window", -3: "FixedRowFFD failed",
          -4: "infeasible layout", -5: "fixed-point overflow", -6: "HIP error",
          -7: "postcondition failed", -8: "unsupported size"}

LEVEL_KERNELS = {0: "workgroup", 1: "wave", 2: "chain", 3: "chain_run"}

EXPORTS = ("routepack_aggregate_demand", "routepack_place_experts", "routepack_pack_rows",
           "routepack_anneal", "routepack_eval_objective", "routepack_select_population",
           "routepack_row_lower_bound", "routepack_fixed_bin_search", "routepack_project_demand",
           "routepack_strerror")
# measurement aid declared in include/routepack_probe.h (not part of the method),
# built as its own library
PROBE_EXPORTS = ("routepack_probe_lds_read",)
PROBE_LIB_PATH = os.path.join(_HERE, "libroutepack_probe.so")


class RoutepackError(RuntimeError):
    def __init__(self, fn, code):
        super().__init__(f"{fn} failed: {code} ({ERRORS.get(code, 'unknown')})")
        self.code = code


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
                ("sweep_offset", C.c_int32), ("init_incumbent", C.c_int32),
                ("level_kernel_ms", C.POINTER(C.c_double)), ("level_kernel", C.POINTER(C.c_int32))]


_lib = None


def load_library():
    """Loads libroutepack.so; raises if it was not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: run __graft_entry__.build() first")
        lib = C.CDLL(LIB_PATH)
        vp, i32, i64, u64 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64
        P = C.POINTER(_Problem)
        lib.routepack_aggregate_demand.argtypes = [P, vp, vp, vp]
        lib.routepack_place_experts.argtypes = [P, vp, vp, vp, vp, vp, vp]
        lib.routepack_project_demand.argtypes = [P, vp, vp, vp, vp, vp, vp]
        lib.routepack_pack_rows.argtypes = [P, vp, vp, u64, i32, i32, i32, vp, vp, vp, vp, vp, vp]
        lib.routepack_anneal.argtypes = [P, vp, vp, i32, i32, vp, C.POINTER(_AnnealParams), vp, vp,
                                         vp, vp, vp, vp]
        lib.routepack_eval_objective.argtypes = [P, vp, vp, i32, i32, vp, vp, vp, vp, vp, vp, vp]
        lib.routepack_select_population.argtypes = [P, vp, vp, i32, i32, vp, vp, u64, i32, vp, vp, vp]
        lib.routepack_row_lower_bound.argtypes = [P, vp, C.POINTER(C.c_int32), C.POINTER(C.c_int64), vp]
        lib.routepack_fixed_bin_search.argtypes = [P, vp, i32, i64, C.POINTER(C.c_int32), C.POINTER(C.c_int64), vp,
                                                   vp]
        lib.routepack_strerror.argtypes = [C.c_int]
        lib.routepack_strerror.restype = C.c_char_p
        for f in EXPORTS:
            if f != "routepack_strerror":
                getattr(lib, f).restype = C.c_int
        _lib = lib
    return _lib


class Problem:
    """Problem description (mirrors routepack_problem)."""

    def __init__(self, n_samples, n_layers, n_experts, top_k, n_ranks, n_dp, n_edp, dp_to_edp,
                 capacity, alpha_fp, beta_fp, frac_bits=12, min_rows=1):
        self.dp_to_edp = np.ascontiguousarray(dp_to_edp, dtype=np.int32)
        self.alpha_fp = np.ascontiguousarray(alpha_fp, dtype=np.int64)
        self.beta_fp = np.ascontiguousarray(beta_fp, dtype=np.int64)
        self.n_samples, self.n_layers, self.n_experts = int(n_samples), int(n_layers), int(n_experts)
        self.top_k, self.n_ranks, self.n_dp, self.n_edp = int(top_k), int(n_ranks), int(n_dp), int(n_edp)
        self.capacity, self.frac_bits, self.min_rows = int(capacity), int(frac_bits), int(min_rows)
        self._c = _Problem(self.n_samples, self.n_layers, self.n_experts, self.top_k, self.n_ranks,
                           self.n_dp, self.n_edp,
                           self.dp_to_edp.ctypes.data_as(C.POINTER(C.c_int32)), self.capacity,
                           len(self.alpha_fp), self.alpha_fp.ctypes.data_as(C.POINTER(C.c_int64)),
                           self.beta_fp.ctypes.data_as(C.POINTER(C.c_int64)), self.frac_bits,
                           self.min_rows)

    @classmethod
    def from_dict(cls, d):
        return cls(**d)

    @property
    def ref(self):
        return C.byref(self._c)


def _torch():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("the RoutePack HIP path needs a GPU (torch.cuda.is_available() is False)")
    return torch


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream():
    torch = _torch()
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _check(fn, rc):
    if rc != 0:
        raise RoutepackError(fn, rc)


def _dev(x, dtype):
    torch = _torch()
    if isinstance(x, torch.Tensor):
        assert x.is_cuda and x.dtype == dtype and x.is_contiguous(), (x.device, x.dtype)
        return x
    return torch.as_tensor(np.ascontiguousarray(x), device="cuda").to(dtype).contiguous()


def aggregate_demand(prob: Problem, demand):
    """agg[l][e] = sum_i demand[i][l][e] (int64), computed on the GPU."""
    torch = _torch()
    lib = load_library()
    d = _dev(demand, torch.int32)
    agg = torch.empty((prob.n_layers, prob.n_experts), dtype=torch.int64, device="cuda")
    _check("routepack_aggregate_demand", lib.routepack_aggregate_demand(prob.ref, _ptr(d), _ptr(agg), _stream()))
    return agg


def aggregate_demand_noalloc(prob: Problem, demand, out=None):
    """aggregate_demand through routepack_aggregate_demand_noalloc: the
    library allocates nothing (its partials live in a fixed device array);
    `out` (int64 [L][E] on the device) receives the result when given."""
    torch = _torch()
    lib = load_library()
    d = _dev(demand, torch.int32)
    agg = out if out is not None else torch.empty((prob.n_layers, prob.n_experts), dtype=torch.int64,
                                                  device="cuda")
    _check("routepack_aggregate_demand_noalloc",
           lib.routepack_aggregate_demand_noalloc(prob.ref, _ptr(d), _ptr(agg), _stream()))
    return agg


def place_experts(prob: Problem, agg, demand=None):
    """Layer-local LPT: returns (slot_of [L][E], rank_load [L][P], q [N][L][P] or None)."""
    torch = _torch()
    lib = load_library()
    a = _dev(agg, torch.int64)
    slot = torch.empty((prob.n_layers, prob.n_experts), dtype=torch.int32, device="cuda")
    load = torch.empty((prob.n_layers, prob.n_ranks), dtype=torch.int64, device="cuda")
    d = None if demand is None else _dev(demand, torch.int32)
    q = None
    if d is not None:
        q = torch.empty((prob.n_samples, prob.n_layers, prob.n_ranks), dtype=torch.int32, device="cuda")
    _check("routepack_place_experts", lib.routepack_place_experts(prob.ref, _ptr(a), _ptr(slot), _ptr(load),
                                                                   _ptr(d), _ptr(q), _stream()))
    return slot, load, q


def project_demand(prob: Problem, agg, slot_of, demand=None):
    """A given placement: returns (rank_load [L][P], q [N][L][P] or None)."""
    torch = _torch()
    lib = load_library()
    a = _dev(agg, torch.int64)
    s = _dev(slot_of, torch.int32)
    load = torch.empty((prob.n_layers, prob.n_ranks), dtype=torch.int64, device="cuda")
    d = None if demand is None else _dev(demand, torch.int32)
    q = None
    if d is not None:
        q = torch.empty((prob.n_samples, prob.n_layers, prob.n_ranks), dtype=torch.int32, device="cuda")
    _check("routepack_project_demand", lib.routepack_project_demand(prob.ref, _ptr(a), _ptr(s), _ptr(load),
                                                                     _ptr(d), _ptr(q), _stream()))
    return load, q


def pack_rows(prob: Problem, lengths, q, seed, n_trials, width, pop):
    """Row-count search and seed population; returns a dict."""
    torch = _torch()
    lib = load_library()
    t = _dev(lengths, torch.int32)
    qq = _dev(q, torch.int32)
    popl = torch.empty((pop, prob.n_samples), dtype=torch.int32, device="cuda")
    sc = torch.empty((pop, 3), dtype=torch.int64, device="cuda")
    r_star, cert = C.c_int32(0), C.c_int32(0)
    info = (C.c_int32 * 3)()
    rc = lib.routepack_pack_rows(prob.ref, _ptr(t), _ptr(qq), C.c_uint64(seed), n_trials, width, pop,
                                 C.byref(r_star), C.byref(cert), _ptr(popl), _ptr(sc), info, _stream())
    _check("routepack_pack_rows", rc)
    return dict(r_star=r_star.value, certified=bool(cert.value), population=popl, scores=sc,
                r_lb=info[0], n_distinct=info[1], n_trials_ok=info[2])


def anneal(prob: Problem, lengths, q, n_rows, population, temperatures, steps_per_sweep, seed,
           t_next=0.0, sweep_offset=0, p_guide_u32=0xCCCCCCCD, rho_u32=0x40000000,
           best_layout=None, best_score=None, want_trace=True, want_parents=True, want_steps=False,
           inplace=False, kernel_times=False):
    """Population annealing; returns dict(population, best_layout, best_score, trace, parents, steps)."""
    torch = _torch()
    lib = load_library()
    t = _dev(lengths, torch.int32)
    qq = _dev(q, torch.int32)
    popl = _dev(population, torch.int32)
    if not inplace:
        popl = popl.clone()
    P, N = popl.shape
    temps = np.ascontiguousarray(temperatures, dtype=np.float64)
    ns = len(temps)
    init = best_layout is None
    bl = torch.zeros(N, dtype=torch.int32, device="cuda") if init else _dev(best_layout, torch.int32).clone()
    bs = torch.zeros(3, dtype=torch.int64, device="cuda") if init else _dev(best_score, torch.int64).clone()
    trace = torch.empty((ns, P, 8), dtype=torch.int64, device="cuda") if want_trace else None
    parents = torch.empty((ns, P), dtype=torch.int32, device="cuda") if want_parents else None
    steps = torch.empty((ns, P, steps_per_sweep), dtype=torch.uint8, device="cuda") if want_steps else None
    kms = np.zeros(max(ns, 1), dtype=np.float64) if kernel_times else None
    used = C.c_int32(-1)
    ap = _AnnealParams(ns, steps_per_sweep, temps.ctypes.data_as(C.POINTER(C.c_double)), float(t_next),
                       p_guide_u32, rho_u32, seed, sweep_offset, 1 if init else 0,
                       kms.ctypes.data_as(C.POINTER(C.c_double)) if kms is not None else None,
                       C.pointer(used))
    rc = lib.routepack_anneal(prob.ref, _ptr(t), _ptr(qq), n_rows, P, _ptr(popl), C.byref(ap), _ptr(bl),
                              _ptr(bs), _ptr(trace), _ptr(parents), _ptr(steps), _stream())
    _check("routepack_anneal", rc)
    return dict(population=popl, best_layout=bl, best_score=bs, trace=trace, parents=parents, steps=steps,
                level_kernel_ms=None if kms is None else kms[:ns],
                level_kernel=LEVEL_KERNELS.get(used.value))


def eval_objective(prob: Problem, lengths, q, n_rows, layouts, rank_load=None, want_J=False,
                   want_diag=False):
    """Exact scores, status and optional J / diagnostics of many layouts."""
    torch = _torch()
    lib = load_library()
    t = _dev(lengths, torch.int32)
    qq = _dev(q, torch.int32)
    lay = _dev(layouts, torch.int32)
    if lay.dim() == 1:
        lay = lay.unsqueeze(0)
    n = lay.shape[0]
    sc = torch.empty((n, 3), dtype=torch.int64, device="cuda")
    st = torch.empty(n, dtype=torch.int32, device="cuda")
    J = torch.empty((n, n_rows * prob.n_edp), dtype=torch.int64, device="cuda") if want_J else None
    dg = torch.empty((n, 8), dtype=torch.float64, device="cuda") if want_diag else None
    rl = None if rank_load is None else _dev(rank_load, torch.int64)
    rc = lib.routepack_eval_objective(prob.ref, _ptr(t), _ptr(qq), n_rows, n, _ptr(lay), _ptr(sc), _ptr(st),
                                      _ptr(J), _ptr(dg), _ptr(rl), _stream())
    _check("routepack_eval_objective", rc)
    return dict(scores=sc, status=st, J=J, diag=dg)


_probe_lib = None


def load_probe_library():
    """Loads libroutepack_probe.so (the LDS read-bandwidth probe)."""
    global _probe_lib
    if _probe_lib is None:
        if not os.path.exists(PROBE_LIB_PATH):
            raise RuntimeError(f"{PROBE_LIB_PATH} is missing: run __graft_entry__.build() first")
        lib = C.CDLL(PROBE_LIB_PATH)
        lib.routepack_probe_lds_read.argtypes = [C.c_int32, C.c_int32, C.c_void_p, C.POINTER(C.c_double),
                                                 C.POINTER(C.c_int64), C.c_void_p]
        lib.routepack_probe_lds_read.restype = C.c_int
        _probe_lib = lib
    return _probe_lib


def probe_lds_read(n_workgroups=2048, reps=8192):
    """LDS read bandwidth of this device (routepack_probe_lds_read): returns
    (bytes read, launch ms).  A measurement aid, not part of the method."""
    torch = _torch()
    lib = load_probe_library()
    sink = torch.empty(n_workgroups * 256, dtype=torch.int32, device="cuda")
    ms, nbytes = C.c_double(0.0), C.c_int64(0)
    _check("routepack_probe_lds_read",
           lib.routepack_probe_lds_read(int(n_workgroups), int(reps), _ptr(sink), C.byref(ms), C.byref(nbytes),
                                        _stream()))
    return int(nbytes.value), float(ms.value)


def select_population(prob: Problem, lengths, q, n_rows, candidates, primary, seed, pop_size=0):
    """QualityDiversitySelect (routepack_select_population): the selection
    order of the candidates and, when pop_size > 0, the population they fill."""
    torch = _torch()
    lib = load_library()
    t = _dev(lengths, torch.int32)
    qq = _dev(q, torch.int32) if q is not None else None
    cand = _dev(candidates, torch.int32)
    s0 = _dev(primary, torch.int64)
    M = cand.shape[0]
    order = torch.empty(M, dtype=torch.int32, device="cuda")
    pop = torch.empty((pop_size, prob.n_samples), dtype=torch.int32, device="cuda") if pop_size > 0 else None
    _check("routepack_select_population",
           lib.routepack_select_population(prob.ref, _ptr(t), _ptr(qq), int(n_rows), int(M), _ptr(cand), _ptr(s0),
                                           C.c_uint64(seed), int(pop_size), _ptr(order), _ptr(pop), _stream()))
    return {"order": order, "population": pop}


def row_lower_bound(prob: Problem, lengths):
    """(R_bound, K_bound) of routepack_row_lower_bound: R* is minimal when it
    equals R_bound."""
    torch = _torch()
    lib = load_library()
    t = _dev(lengths, torch.int32)
    r, k = C.c_int32(0), C.c_int64(0)
    _check("routepack_row_lower_bound", lib.routepack_row_lower_bound(prob.ref, _ptr(t), C.byref(r), C.byref(k),
                                                                      _stream()))
    return int(r.value), int(k.value)


def fixed_bin_search(prob: Problem, lengths, n_rows, node_budget):
    """routepack_fixed_bin_search: (status, nodes, layout or None); status 1
    feasible, 0 infeasible, 2 unknown."""
    torch = _torch()
    lib = load_library()
    t = _dev(lengths, torch.int32)
    lay = torch.full((prob.n_samples,), -1, dtype=torch.int32, device="cuda")
    st, nodes = C.c_int32(0), C.c_int64(0)
    _check("routepack_fixed_bin_search",
           lib.routepack_fixed_bin_search(prob.ref, _ptr(t), int(n_rows), int(node_budget), C.byref(st),
                                          C.byref(nodes), _ptr(lay), _stream()))
    return int(st.value), int(nodes.value), (lay if st.value == 1 else None)
