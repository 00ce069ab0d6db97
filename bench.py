#!/usr/bin/env python3
"""Benchmark of the RoutePack planner hot path on one MI355X.

One step is one pass of the whole path over one synthetic optimizer-step
window already resident in HBM: demand aggregation, LPT placement and rank
projection, row packing with the seed population, and population annealing
over the full temperature schedule (plus the library's own validation of x*).

Workload (default): the mid window -- 4096 samples with lognormal lengths
(median 4096, sigma 1.0, clipped to [128, 32768]), 24 MoE layers of 256
experts, top-8 routing with a Zipf(1.2) profile drifting 10% per layer,
16 EP ranks, 8 DP slots in one EDP shard, cap 65536 tokens; population 1024,
2000 levels of 256 proposals.

Metric: annealing move-evals/s = evaluated (feasible) proposals of all
levels and members, over the wall time of the steps.  The JSON line also
carries the roofline of the dominant kernel (the annealing level kernel) from HIP events
on the library's stream, and the CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# Sources of each level kernel (its own file plus the shared annealing code).
LEVEL_KERNEL_FILES = {
    "chain_run": "rp_anneal_chain.hip",
    "chain": "rp_anneal_chain.hip",
    "wave": "rp_anneal_wave.hip",
    "workgroup": "rp_anneal.hip",
}


def kernel_sources(kernel):
    files = sorted({LEVEL_KERNEL_FILES[kernel], "rp_anneal.h", "rp_anneal.hip", "rp_device.h"})
    return [os.path.join(ROOT, "paper_2608_12146_amd", "csrc", f) for f in files]


def config_tag(window, G=1, S=1):
    """Name of a workload in profile file names: the window, plus the EDP
    shard and stage counts when they are not 1."""
    return window + (f"_g{G}" if G != 1 else "") + (f"_s{S}" if S != 1 else "")


def pmc_file(kernel, window):
    return os.path.join(ROOT, "profiles", f"anneal_{kernel}_{window}_pmc.txt")


def lds_file(kernel, window):
    return os.path.join(ROOT, "profiles", f"anneal_{kernel}_{window}_lds.txt")


def _code_text(src: str) -> str:
    """The source with // comments and blank lines removed (comment edits do
    not change the kernel the counters were taken on)."""
    out = []
    for line in src.splitlines():
        i = line.find("//")
        if i >= 0 and line.count('"', 0, i) % 2 == 0:
            line = line[:i]
        line = line.rstrip()
        if line:
            out.append(line)
    return "\n".join(out)


def kernel_source_hash(kernel) -> str:
    """SHA-256 of the kernel's sources (code only) and of the flags the
    .hip ones compile with."""
    from paper_2608_12146_amd import build as B
    h = hashlib.sha256()
    for f in kernel_sources(kernel):
        with open(f, encoding="utf-8") as fh:
            h.update(_code_text(fh.read()).encode())
        if f.endswith(".hip"):
            h.update(" ".join(B.flags_for(f)).encode())
    return h.hexdigest()[:16]


def _read_profile(path, kernel):
    """key: value lines of a counter summary, if taken on this kernel's sources."""
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256_16") != kernel_source_hash(kernel):
        return None
    return kv


def read_pmc(kernel, window):
    """Counter-derived HBM traffic per dispatch, if taken on this kernel's sources."""
    kv = _read_profile(pmc_file(kernel, window), kernel)
    try:
        return float(kv["hbm_bytes_per_dispatch"]) if kv else None
    except (KeyError, ValueError):
        return None


def read_lds(kernel, window, launch_ms):
    """LDS bytes per dispatch from the counters (if taken on this kernel's
    sources) over the live launch time, against the LDS peak (256 B per clock
    per CU, as the counters show, at 2.4 GHz); the LDS probe's sustained rate
    rides along."""
    kv = _read_profile(lds_file(kernel, window), kernel)
    if not kv:
        return None
    try:
        nbytes = float(kv["lds_load_bytes_per_dispatch"]) + float(kv["lds_store_bytes_per_dispatch"])
        peak = float(kv["lds_read_peak_gbs"])
        achieved = nbytes / (launch_ms * 1e6)
        return {"achieved": achieved, "peak": peak, "unit": "GB/s", "frac": achieved / peak,
                "bytes_per_launch": nbytes, "probe_gbs": float(kv["lds_probe_gbs"]),
                "busy_frac": float(kv["lds_busy_frac"]),
                "bank_conflict_cycles_frac": float(kv["lds_bank_conflict_frac"])}
    except (KeyError, ValueError, ZeroDivisionError):
        return None


def workload_text(w, G, S=1):
    return (f"{w.name} window: {w.n} samples, {w.n_layers} layers x {w.n_experts} experts top-{w.top_k}, "
            f"{w.n_ranks} EP ranks, {w.n_dp} DP slots in {G} EDP shard(s), cap {w.capacity}, "
            + ("two attention stages (linear + quadratic), " if S == 2 else "")
            + f"population {w.pop}, {w.levels} levels x 256 proposals")


def copy_probe():
    """A plain copy of known size, for scaling FETCH_SIZE / WRITE_SIZE."""
    import torch
    n = 256 << 20
    src = torch.ones(n // 4, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": n, "dispatches": 5}))


def lds_probe():
    """LDS read bandwidth of this device: four launches of the library's LDS
    streaming probe (the first a warm-up); the fastest timed one is reported."""
    import paper_2608_12146_amd as rp
    rp.probe_lds_read(256, 64)
    runs = [rp.probe_lds_read() for _ in range(3)]
    nbytes, ms = min(runs, key=lambda r: r[1])
    print(json.dumps({"lds_probe_bytes": nbytes, "ms": ms, "GB/s": nbytes / ms / 1e6, "dispatches": 4}))


def occupancy(kernel, pop):
    """Launch shape of the level kernel at this population on the 256 CUs
    (1024 SIMDs): the chain kernels run one wave per member and spread the
    members over the CUs, at most four per workgroup (the member state fills
    the LDS)."""
    if kernel in ("chain_run", "chain"):
        mpw = max(1, min(4, -(-pop // 256)))  # members per workgroup
        wgs = -(-pop // mpw)
        per_cu = -(-wgs // 256)
        return {"workgroups": wgs, "waves_per_workgroup": mpw, "workgroups_per_cu": per_cu,
                "waves_per_simd": -(-(mpw * per_cu) // 4), "waves_per_member": 1}
    return None


def demand_stream(reps=10):
    """The HBM stream of the path's first steps at the largest window shape
    (32768 samples, 64 layers x 512 experts, 64 ranks: 4 GiB of int32
    demand, seeded random counts): routepack_aggregate_demand (algorithmic
    bytes N L E 4 read + L E 8 written) and routepack_place_experts (LPT and
    the projection: N L E 4 read + N L P 4 written), each timed with HIP
    events on the library's stream over `reps` calls."""
    import torch
    import paper_2608_12146_amd as rp
    N, L, E, P = 32768, 64, 512, 64
    g = torch.Generator(device="cuda")
    g.manual_seed(2608)
    d = torch.randint(0, 64, (N, L, E), dtype=torch.int32, device="cuda", generator=g)
    prob = rp.Problem(N, L, E, 8, P, 1, 1, [0], 1 << 20, [4096], [1])
    agg = rp.aggregate_demand(prob, d)
    ok = bool(torch.equal(agg, d.sum(dim=0, dtype=torch.int64)))
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    s.record()
    for _ in range(reps):
        rp.aggregate_demand(prob, d)
    e.record()
    torch.cuda.synchronize()
    ms_a = s.elapsed_time(e) / reps
    rp.place_experts(prob, agg, d)
    torch.cuda.synchronize()
    s.record()
    for _ in range(reps):
        rp.place_experts(prob, agg, d)
    e.record()
    torch.cuda.synchronize()
    ms_p = s.elapsed_time(e) / reps
    ba, bp = N * L * E * 4 + L * E * 8, N * L * E * 4 + N * L * P * 4
    del d
    torch.cuda.empty_cache()
    return {"shape": {"samples": N, "layers": L, "experts": E, "ranks": P},
            "aggregate": {"ms_per_call": ms_a, "bytes": ba, "achieved_gbs": ba / ms_a / 1e6,
                          "frac": ba / ms_a / 1e6 / HBM_PEAK_GBS, "eq_torch_sum": ok},
            "place_and_project": {"ms_per_call": ms_p, "bytes": bp, "achieved_gbs": bp / ms_p / 1e6,
                                  "frac": bp / ms_p / 1e6 / HBM_PEAK_GBS}}


DIAG_KEYS = ("cv_global", "s_ep", "t_ep", "eta_ep", "attention", "joint")


def _diag(d):
    """eval_objective's diagnostics as named metrics: CV_global, S_EP, T_EP,
    eta_EP, the attention sum and the joint max_g U (normalised by C)."""
    return {k: float(v) for k, v in zip(DIAG_KEYS, (d[0], d[1], d[2], d[3], d[4], d[5]))}


def compare_planners(rp, w, pd, levels, t_first=None, t_last=None):
    """Three planners on one window, all on the GPU path, scored by the same
    diagnostics (Sec. 5.3): baseline = identity placement pi_l(e) = e with the
    length-only FFD layout; reorder = LPT placement with that FFD layout;
    routepack = LPT placement, Alg. 2 seeds and annealing for `levels` levels
    of the window's schedule.  The FFD layout is x_length of a two-trial
    packing: the later of its one or two distinct seeds (x_paired is kept
    only when strictly better, and the population is ordered by score)."""
    import torch
    import synth
    from synth import windows as W
    prob = rp.Problem.from_dict(pd)
    demand = torch.as_tensor(w.demand, device="cuda")
    lengths = torch.as_tensor(w.lengths, device="cuda")
    agg = rp.aggregate_demand(prob, demand)
    ident = torch.arange(w.n_experts, dtype=torch.int32, device="cuda").repeat(w.n_layers, 1)
    g_id, q_id = rp.project_demand(prob, agg, ident, demand)
    _, g_lpt, q = rp.place_experts(prob, agg, demand)
    ffd = rp.pack_rows(prob, lengths, q, w.seed_pack, 2, 1, 2)
    R = ffd["r_star"]
    x_ffd = ffd["population"][ffd["n_distinct"] - 1]
    pk = rp.pack_rows(prob, lengths, q, w.seed_pack, W.N_TRIALS, W.CHOICE_WIDTH, w.pop)
    temps = synth.anneal_temperatures(w.levels, t_first or W.T_FIRST, t_last or W.T_LAST)[:levels]
    an = rp.anneal(prob, lengths, q, R, pk["population"], temps, W.STEPS_PER_LEVEL, w.seed_anneal,
                   want_trace=False, want_parents=False)
    rows = {}
    for name, qq, g, x in (("baseline", q_id, g_id, x_ffd), ("reorder", q, g_lpt, x_ffd),
                           ("routepack", q, g_lpt, an["best_layout"])):
        ev = rp.eval_objective(prob, lengths, qq, R, x, rank_load=g, want_diag=True)
        assert int(ev["status"][0]) == 0
        rows[name] = _diag(ev["diag"][0].cpu().numpy())
    return {"window": w.name, "n_rows": R, "levels": levels, **rows,
            "layouts": {"ffd": x_ffd.cpu().numpy(), "routepack": an["best_layout"].cpu().numpy()}}


def compare(windows, levels, t_first=None, t_last=None):
    """One JSON line per window: the three planners' metrics and the change
    from each to the next (X3: CV_global under LPT; X4: FFD to annealing)."""
    import paper_2608_12146_amd as rp
    import synth
    for name in windows:
        print(f"[compare] {name}: generating", file=sys.stderr, flush=True)
        w = synth.make_window(name)
        pd = synth.window_problem(w)
        t1 = time.perf_counter()
        r = compare_planners(rp, w, pd, levels or w.levels, t_first, t_last)
        r["temperatures"] = [t_first or synth.windows.T_FIRST, t_last or synth.windows.T_LAST]
        r.pop("layouts")
        b, o, g = r["baseline"], r["reorder"], r["routepack"]
        r["change"] = {
            "cv_global_lpt": o["cv_global"] / b["cv_global"] - 1.0 if b["cv_global"] else None,
            **{f"{k}_anneal": g[k] / o[k] - 1.0 if o[k] else None for k in DIAG_KEYS[1:]},
        }
        r["seconds"] = time.perf_counter() - t1
        print(f"[compare] {name}: {r['seconds']:.1f} s", file=sys.stderr, flush=True)
        print(json.dumps(r), flush=True)


def cpu_model():
    """The host CPU's model name (/proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--window", default="mid")
    ap.add_argument("--edp", type=int, default=1, help="EDP shards G (contiguous slot blocks)")
    ap.add_argument("--stages", type=int, default=1, choices=(1, 2),
                    help="attention stages: 1, or 2 (a linear and a quadratic stage)")
    ap.add_argument("--levels", type=int, default=None, help="levels (default: the window's schedule)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-levels", type=int, default=None,
                    help="levels the oracle runs after the timed region (default: the whole schedule, "
                         "whose trajectory is then compared with the last timed step's)")
    ap.add_argument("--no-extra-windows", action="store_true",
                    help="skip the short heavy-tail and stress runs reported under extra_windows")
    ap.add_argument("--print-maps", action="store_true",
                    help="print /proc/self/maps to stderr before exiting (to attribute exit-time faults)")
    ap.add_argument("--copy-probe", action="store_true")
    ap.add_argument("--lds-probe", action="store_true")
    ap.add_argument("--demand-probe", action="store_true",
                    help="only the aggregation / projection HBM stream at the largest window shape")
    ap.add_argument("--compare", default=None, metavar="WINDOWS",
                    help="comma-separated windows: baseline / reorder / routepack metrics instead of the bench")
    ap.add_argument("--t-first", type=float, default=None, help="--compare: first temperature of the schedule")
    ap.add_argument("--t-last", type=float, default=None, help="--compare: last temperature of the schedule")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the planner path is "
              "single-GPU; sharding the population across GPUs is not implemented", file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_probe:
        copy_probe()
        return
    if args.lds_probe:
        lds_probe()
        return
    if args.demand_probe:
        print(json.dumps(demand_stream()), flush=True)
        return
    if args.compare:
        compare(args.compare.split(","), args.levels, args.t_first, args.t_last)
        return

    import paper_2608_12146_amd as rp
    import synth
    from synth import windows as W

    w = synth.make_window(args.window, edp=args.edp)
    pd = synth.window_problem(w, stages=args.stages)
    prob = rp.Problem.from_dict(pd)
    levels = args.levels or w.levels
    temps = synth.anneal_temperatures(w.levels)[:levels]
    K = W.STEPS_PER_LEVEL
    demand = torch.as_tensor(w.demand, device="cuda")
    lengths = torch.as_tensor(w.lengths, device="cuda")
    torch.cuda.synchronize()

    def step():
        agg = rp.aggregate_demand(prob, demand)
        slot, load, q = rp.place_experts(prob, agg, demand)
        pk = rp.pack_rows(prob, lengths, q, w.seed_pack, W.N_TRIALS, W.CHOICE_WIDTH, w.pop)
        an = rp.anneal(prob, lengths, q, pk["r_star"], pk["population"], temps, K, w.seed_anneal,
                       want_parents=False, kernel_times=True)
        return q, load, pk, an

    def progress(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    progress(f"{workload_text(w, args.edp, args.stages)}; levels {levels}")
    for k in range(args.warmup):
        t1 = time.perf_counter()
        step()
        torch.cuda.synchronize()
        progress(f"warmup {k} {time.perf_counter() - t1:.2f} s")
    evals = acc = 0
    kernel_ms = []
    level_kernel = None
    t0 = time.perf_counter()
    for _ in range(args.steps):
        q, load, pk, an = step()
        tr = an["trace"]
        evals += int(tr[:, :, 7].sum().item())
        acc += int(tr[:, :, 6].sum().item())
        kernel_ms.append(an["level_kernel_ms"])
        level_kernel = an["level_kernel"]
        progress(f"step done at {time.perf_counter() - t0:.2f} s")
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    attempted = args.steps * levels * w.pop * K

    # Roofline of the level kernel: algorithmic global bytes of an evaluated
    # move are the moved samples' q rows (2 L P int32 for a swap, L P for a
    # relocation), expected (2 - rho) L P 4 bytes at relocation rate rho.
    rho = W.RHO_U32 / 2.0**32
    bytes_per_eval = (2.0 - rho) * w.n_layers * w.n_ranks * 4
    kms = np.concatenate(kernel_ms)
    k_sec = float(kms.sum()) / 1e3
    # the whole-schedule kernel is one launch per step; the others one per level
    launches = args.steps * (1 if level_kernel == "chain_run" else levels)
    achieved = evals * bytes_per_eval / k_sec / 1e9
    tag = config_tag(args.window, args.edp, args.stages)
    traffic = read_pmc(level_kernel, tag)
    lds = read_lds(level_kernel, tag, float(kms.sum()) / launches)

    # Objective == oracle, outside the timed region: the oracle's seed
    # population and rescoring of the GPU's x*; below, the oracle's run of
    # the schedule against the last timed step's trajectory.
    import oracle as O
    pb = O.Problem.from_dict(pd)
    qn = q.cpu().numpy()
    st, s_or, _, _ = O.score(pb, w.lengths, qn, pk["r_star"], an["best_layout"].cpu().numpy())
    score_ok = st == 0 and s_or.tolist() == an["best_score"].cpu().tolist()
    opk = O.pack_rows(pb, w.lengths, qn, w.seed_pack, W.N_TRIALS, W.CHOICE_WIDTH, w.pop)
    pack_ok = (opk["r_star"] == pk["r_star"]
               and bool(np.array_equal(opk["population"], pk["population"].cpu().numpy()))
               and bool(np.array_equal(opk["scores"], pk["scores"].cpu().numpy())))
    progress(f"parity: x* rescored {score_ok}, pack {pack_ok}")

    # QualityDiversitySelect on the window's canonical-distinct seeds: its own
    # timing (the default step keeps the (score, discovery) seed order) and
    # its order against the oracle's.
    from oracle import qds
    M = int(pk["n_distinct"])
    cands = pk["population"][:M]
    s0 = pk["scores"][:M, 0].contiguous()
    sel_ms = []
    for _ in range(6):
        t1 = time.perf_counter()
        sel = rp.select_population(prob, lengths, q, pk["r_star"], cands, s0, w.seed_pack, pop_size=w.pop)
        sel_ms.append((time.perf_counter() - t1) * 1e3)
    want = qds.select(pb, w.lengths, qn, opk["r_star"], opk["population"][:M], opk["scores"][:M, 0], w.seed_pack)
    select = {"candidates": M, "ms_per_call": float(np.median(sel_ms[1:])),
              "order_eq_oracle": sel["order"].cpu().tolist() == want.tolist()}
    progress(f"select_population: {M} candidates, {select['ms_per_call']:.3f} ms, "
             f"order == oracle {select['order_eq_oracle']}")

    # The row-count lower bound (volume, cardinality, Martello-Toth L2): R*
    # is the minimum when it reaches it.
    from oracle import bounds
    rb_ms = []
    for _ in range(6):
        t1 = time.perf_counter()
        rb = rp.row_lower_bound(prob, lengths)
        rb_ms.append((time.perf_counter() - t1) * 1e3)
    row_bound = {"r_bound": rb[0], "cell_bound": rb[1], "ms_per_call": float(np.median(rb_ms[1:])),
                 "eq_oracle": rb == bounds.row_lower_bound(w.lengths, w.capacity, w.n_dp),
                 "r_star_minimal": pk["r_star"] == rb[0]}

    # The fixed-bin search at the bound's row count: feasible there means the
    # bound is R_min whatever FFD found.
    from oracle import fixedbin
    fb_ms = []
    for _ in range(4):
        t1 = time.perf_counter()
        fb = rp.fixed_bin_search(prob, lengths, rb[0], 10 ** 6)
        fb_ms.append((time.perf_counter() - t1) * 1e3)
    fw = fixedbin.search(w.lengths, w.capacity, rb[0] * w.n_dp, 10 ** 6)
    search = {"n_rows": rb[0], "status": fb[0], "nodes": fb[1], "ms_per_call": float(np.median(fb_ms[1:])),
              "eq_oracle": fb[:2] == fw[:2] and (fb[2] is None) == (fw[2] is None)
              and (fb[2] is None or np.array_equal(fb[2].cpu().numpy(), fw[2]))}
    progress(f"fixed_bin_search at R={rb[0]}: status {fb[0]}, {fb[1]} nodes, {search['ms_per_call']:.3f} ms, "
             f"== oracle {search['eq_oracle']}")
    dstream = demand_stream()
    progress(f"demand stream at 32768 x 64 x 512: aggregate {dstream['aggregate']['achieved_gbs']:.0f} GB/s, "
             f"place+project {dstream['place_and_project']['achieved_gbs']:.0f} GB/s")
    # The oracle (the paper's host-worker design: P_pop chains on a pool of
    # threads, a barrier and a resampling per level) on the same window and
    # schedule, timed; with the whole schedule its trace of every level, its
    # final population, x* and best score must equal the last timed step's.
    cpu, traj = None, None
    if not args.no_cpu_baseline:
        host_cpus = len(os.sched_getaffinity(0))
        threads = max(1, min(16, host_cpus))
        nl = levels if args.cpu_levels is None else max(1, min(args.cpu_levels, levels))
        progress(f"cpu baseline: the oracle over levels 0-{nl - 1} on {threads} threads")
        tc = time.perf_counter()
        oc = O.anneal(pb, w.lengths, qn, opk["r_star"], opk["population"], temps[:nl], K, w.seed_anneal,
                      t_next=(temps[nl] if nl < len(temps) else 0.0), n_threads=threads,
                      want_parents=False)
        tcpu = time.perf_counter() - tc
        cev = int(oc["trace"][:, :, 7].sum())
        cpu = {"value": cev / tcpu, "unit": "move-evals/s", "cores": threads, "kind": "oracle",
               "host_cpus": host_cpus, "nproc": os.cpu_count(), "cpu_model": cpu_model(),
               "sample": (f"levels 0-{nl - 1} of the same schedule (of {levels}), population {w.pop}, "
                          f"{cev} evaluated moves in {tcpu:.1f} s on {threads} threads "
                          f"({host_cpus} host CPUs available to the process)")}
        gt = an["trace"].cpu().numpy()
        traj = {"levels_compared": nl, "trace_eq_oracle": bool(oc["rc"] == 0 and np.array_equal(gt[:nl], oc["trace"]))}
        if nl == levels:
            traj["final_population_eq_oracle"] = bool(np.array_equal(an["population"].cpu().numpy(),
                                                                      oc["population"]))
            traj["x_star_eq_oracle"] = bool(np.array_equal(an["best_layout"].cpu().numpy(), oc["best_layout"]))
            traj["best_score_eq_oracle"] = an["best_score"].cpu().tolist() == oc["best_score"].tolist()
        progress(f"oracle: {cev} evaluated moves in {tcpu:.1f} s; trajectory == GPU {traj}")

    extra = None
    if not args.no_extra_windows and args.window == "mid":
        extra = {}
        for name, nl in (("heavy", 20), ("stress", 20)):
            progress(f"extra window {name}: {nl} levels")
            extra[name] = window_short_run(name, nl)
            progress(f"  {extra[name]['kernel']}: {extra[name]['move_evals_per_s_kernel']:.3e} move-evals/s "
                     f"(kernel), roofline {extra[name]['roofline']['frac']:.4f}, parity {extra[name]['parity']}")

    out = {
        "metric": "anneal move-evals/sec; objective==oracle; % HBM/LDS roofline",
        "value": evals / dt,
        "unit": "move-evals/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": dt / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {"workload": workload_text(w, args.edp, args.stages), "levels": levels, "proposals_per_level": K},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "kernel": "k_anneal_" + level_kernel, "avg_launch_ms": float(kms.sum()) / launches,
                     "launches": launches, "bytes_per_eval": bytes_per_eval,
                     "algorithmic_bytes_per_launch": evals * bytes_per_eval / launches,
                     "lds": lds, "occupancy": occupancy(level_kernel, w.pop)},
        "cpu_baseline": cpu,
        "attempted_per_s": attempted / dt,
        "evals_per_step": evals // args.steps,
        "accept_rate": acc / max(evals, 1),
        "parity": {"x_star_rescored_eq_oracle": bool(score_ok), "pack_eq_oracle": bool(pack_ok),
                   "trajectory": traj},
        "select_population": select,
        "row_lower_bound": row_bound,
        "fixed_bin_search": search,
        "demand_stream": dstream,
        "extra_windows": extra,
        "r_star": pk["r_star"],
        "best_score": an["best_score"].cpu().tolist(),
    }
    print(json.dumps(out), flush=True)


def window_short_run(name, levels):
    """The annealing path on another benchmark window for its first `levels`
    levels (full population, the window's own schedule): the level kernel the
    library picks, its rate over the kernel time (HIP events around each
    launch, second of two runs), the HBM roofline fraction by the same
    algorithmic bytes as the main line, and the oracle's check of three
    members' first level and of x*."""
    import torch

    import oracle as O
    import paper_2608_12146_amd as rp
    import synth
    from synth import windows as W
    w = synth.make_window(name)
    pd = synth.window_problem(w)
    prob = rp.Problem.from_dict(pd)
    demand = torch.as_tensor(w.demand, device="cuda")
    lengths = torch.as_tensor(w.lengths, device="cuda")
    agg = rp.aggregate_demand(prob, demand)
    slot, load, q = rp.place_experts(prob, agg, demand)
    del demand
    pk = rp.pack_rows(prob, lengths, q, w.seed_pack, W.N_TRIALS, W.CHOICE_WIDTH, w.pop)
    temps = synth.anneal_temperatures(w.levels)
    K = W.STEPS_PER_LEVEL
    for _ in range(2):
        an = rp.anneal(prob, lengths, q, pk["r_star"], pk["population"], temps[:levels], K, w.seed_anneal,
                       t_next=temps[levels], want_parents=False, kernel_times=True)
        torch.cuda.synchronize()
    tr = an["trace"].cpu().numpy()
    evals = int(tr[:, :, 7].sum())
    k_ms = float(an["level_kernel_ms"].sum())
    bytes_per_eval = (2.0 - W.RHO_U32 / 2.0**32) * w.n_layers * w.n_ranks * 4
    rate = evals / (k_ms / 1e3)
    pb = O.Problem.from_dict(pd)
    qn = q.cpu().numpy()
    ids = np.array([0, w.pop // 2, w.pop - 1], dtype=np.int32)
    oa = O.anneal(pb, w.lengths, qn, pk["r_star"], pk["population"].cpu().numpy()[ids], temps[:1], K,
                  w.seed_anneal, replica_ids=ids)
    st, s_or, _, _ = O.score(pb, w.lengths, qn, pk["r_star"], an["best_layout"].cpu().numpy())
    out = {"workload": workload_text(w, 1), "levels": levels, "kernel": "k_anneal_" + an["level_kernel"],
           "evals": evals, "kernel_ms": k_ms, "move_evals_per_s_kernel": rate,
           "roofline": {"bound": "hbm", "achieved": rate * bytes_per_eval / 1e9, "peak": HBM_PEAK_GBS,
                        "unit": "GB/s", "frac": rate * bytes_per_eval / 1e9 / HBM_PEAK_GBS,
                        "bytes_per_eval": bytes_per_eval},
           "parity": {"level0_sampled_members_eq_oracle": bool(oa["rc"] == 0 and
                                                               np.array_equal(tr[0][ids], oa["trace"][0])),
                      "x_star_rescored_eq_oracle": bool(st == 0 and
                                                        s_or.tolist() == an["best_score"].cpu().tolist())}}
    del q, an, pk
    return out


def release_device_state():
    """Frees what this process holds on the device before the interpreter
    exits: every stream is drained and torch's cached blocks are returned, so
    no device memory is released from static destructors at exit."""
    import gc

    import torch
    gc.collect()
    if torch.cuda.is_available() and torch.cuda.is_initialized():
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        torch.cuda.synchronize()


if __name__ == "__main__":
    main()
    release_device_state()
    if "--print-maps" in sys.argv:
        with open("/proc/self/maps") as f:
            sys.stderr.write(f.read())
        sys.stderr.flush()
