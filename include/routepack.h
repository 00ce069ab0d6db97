/*
 * routepack.h -- C-ABI of the MI355X (gfx950) RoutePack planner hot path.
 *
 * RoutePack (arXiv 2608.12146) plans one optimizer-step window of a MoE RL
 * trainer in three data-parallel stages, each exported here:
 *   1. window demand aggregation and layer-local LPT expert placement
 *      (Sec. 3.3, Alg. 1), plus the per-sample physical-rank demand
 *      (Eq. physical-rank-demand);
 *   2. the smallest feasible number of token-capped execution rows and a
 *      feasible seed population (Eqs. sample-bijection .. min-row-count,
 *      Alg. 2);
 *   3. fixed-row population annealing over the DP layout of those rows
 *      (Alg. 3) under the EDP-shard-aware lexicographic score
 *      (Eqs. cell-token-statistics .. lexicographic-score).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Arrays are C-order and live in DEVICE memory unless marked [host].  The
 *   caller owns every array; the library keeps no pointer to caller memory
 *   after a call's stream work completes.
 * - Scratch: each (device, stream) the library is called on keeps one
 *   scratch arena from the device's stream-ordered memory pool, sized to the
 *   largest scratch a call on that stream has needed and reused by the next
 *   call there (the stream orders the two); arenas are held until the
 *   process ends.  Scratch that does not fit the arena comes from the pool
 *   and goes back to it before the call returns (synchronous calls) or
 *   stream-ordered on `stream` (asynchronous calls).  Arenas are keyed by
 *   the stream handle: synchronize a stream before destroying it if library
 *   work may still be pending on it, since a new stream can take the same
 *   handle and with it the arena.
 * - Work is enqueued on the caller's `stream`.  Calls marked "synchronizes"
 *   wait for that stream before returning.  Results depend on the arguments
 *   only; calls on different streams are independent (each stream has its
 *   own arena; a second thread that calls on a stream while another thread's
 *   call there is still in progress takes its scratch from the pool).
 * - Layout encoding: a layout is int32 [N] holding, for each sample i, its
 *   cell id c = r * D + d (row r in [0, R), DP slot d in [0, D)).  A
 *   row-shard is h = r * G + g with g = dp_to_edp[d].
 * - Fixed point: every cost is an int64 in units of 2^-F raw tokens; the
 *   paper's normalised value is value / (2^F * C).  Score s = (s0, s1, s2) =
 *   (max_g U_g, sum_g U_g, max_{r,g} J), ordered lexicographically.
 * - Every function returns 0 or one of the negative ROUTEPACK_E_* codes;
 *   on an error nothing is guaranteed about output arrays.
 */
#ifndef ROUTEPACK_H
#define ROUTEPACK_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ROUTEPACK_OK             0
#define ROUTEPACK_E_INVALID     -1  /* null pointer, bad size, E % P != 0, bad partition, C <= 0, bad schedule */
#define ROUTEPACK_E_INFEASIBLE  -2  /* some t_i > C, t_i < 1, or floor(N / D) below the row lower bound */
#define ROUTEPACK_E_HEURISTIC   -3  /* FixedRowFFD found no row count <= floor(N / D) */
#define ROUTEPACK_E_LAYOUT      -4  /* an input layout violates Eqs. sample-bijection .. token-capacity */
#define ROUTEPACK_E_OVERFLOW    -5  /* R*G*(A_max + E_max + 1) >= 2^53: scores not exact in int64/double */
#define ROUTEPACK_E_DEVICE      -6  /* a HIP runtime error */
#define ROUTEPACK_E_INTERNAL    -7  /* a postcondition failed (validation of x*, non-regression) */
#define ROUTEPACK_E_UNSUPPORTED -8  /* a size these kernels do not handle (documented per call) */

/* Problem description (Sec. 3.1-3.4).
 * demand a[i][l][e] and lengths t_i are the routing-replay input (Eq.
 * routing-replay-input); D DP slots are partitioned into G EDP shards by
 * dp_to_edp (every shard non-empty); C is the token cap of one cell (Eq.
 * token-capacity); stage s costs alpha_s * sum t + beta_s * sum t^2 raw
 * tokens (Eq. attention-cost-proxy), given at scale 2^frac_bits; min_rows is
 * an optional pipeline lower bound on R (Sec. 3.2), 1 for none. */
typedef struct routepack_problem {
    int32_t n_samples;        /* N >= 1 */
    int32_t n_layers;         /* L >= 0 MoE layers */
    int32_t n_experts;        /* E >= 1 logical experts per layer */
    int32_t top_k;            /* k: informational */
    int32_t n_ranks;          /* P >= 1 physical EP ranks; E % P == 0; H = E / P */
    int32_t n_dp;             /* D >= 1 controller DP slots */
    int32_t n_edp;            /* G in [1, D] EDP shards */
    const int32_t *dp_to_edp; /* [host][D] shard of each slot */
    int64_t capacity;         /* C >= 1 tokens per cell */
    int32_t n_stages;         /* S >= 1 attention stages */
    const int64_t *alpha_fp;  /* [host][S] >= 0, a_s * 2^frac_bits */
    const int64_t *beta_fp;   /* [host][S] >= 0, b_s * 2^frac_bits */
    int32_t frac_bits;        /* F in [0, 30] */
    int32_t min_rows;         /* >= 1 */
} routepack_problem;

/* Window demand aggregation (Sec. 3.3): agg[l][e] = sum_i demand[i][l][e],
 * exact in int64.
 *   demand  int32 [N][L][E]   replayed routing counts, >= 0
 *   agg     int64 [L][E]      out
 * Asynchronous; allocates stream-ordered scratch of one int64 per column of
 * L E and band of at least 64 rows (at most 4096 / ceil(L E / 256) + 1 bands).
 * E_INVALID on null pointers or negative sizes; E_DEVICE when the scratch
 * cannot be allocated. */
int routepack_aggregate_demand(const routepack_problem *prob, const int32_t *demand,
                               int64_t *agg, hipStream_t stream);

/* routepack_aggregate_demand for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments and result; the band partials live in a fixed
 * device array of 2^20 int64 (8 MiB) that the library holds on each device
 * it runs on until the process ends, so the call allocates nothing (the
 * first call on a device looks the array up with hipGetSymbolAddress).
 * Every call on a device shares that array: calls that overlap on one device
 * (on different streams, or from different threads) race and must be
 * serialized by the caller.  Fewer, taller bands are used when the default
 * band grid would not fit the array.  Asynchronous.  E_UNSUPPORTED when
 * L * E > 2^20 (one band of partials would not fit); E_INVALID as
 * routepack_aggregate_demand; E_DEVICE on a HIP error. */
int routepack_aggregate_demand_noalloc(const routepack_problem *prob, const int32_t *demand,
                                       int64_t *agg, hipStream_t stream);

/* Layer-local LPT placement (Alg. 1), every layer independently: experts by
 * (-agg, e), each to the rank with fewer than H experts minimising
 * (G_p, p), taking slot p*H + n_p.  owner(v) = v / H.
 *   agg         int64 [L][E]          window aggregate
 *   slot_of     int32 [L][E]          out: pi_l(e)
 *   rank_load   int64 [L][P]          out: G_{l,p} (Eq. placement-load)
 *   demand      int32 [N][L][E] or NULL
 *   q           int32 [N][L][P] or NULL  out: q[i][l][p] = sum over e with
 *               owner(pi_l(e)) = p of demand[i][l][e] (Eq. physical-rank-demand);
 *               computed only when both demand and q are given.
 * Asynchronous.  E_INVALID on null outputs or E % P != 0. */
int routepack_place_experts(const routepack_problem *prob, const int64_t *agg,
                            int32_t *slot_of, int64_t *rank_load,
                            const int32_t *demand, int32_t *q, hipStream_t stream);

/* Rank loads and projected demand of a given placement (Sec. 3.3, Eqs.
 * placement-load and physical-rank-demand), for a placement the caller keeps
 * instead of LPT's, such as the identity pi_l(e) = e of a planner that does
 * not reorder experts.
 *   agg         int64 [L][E]          window aggregate
 *   slot_of     int32 [L][E]          pi_l(e); each layer a permutation of [0, E)
 *   rank_load   int64 [L][P]          out: G_{l,p}
 *   demand, q   as in routepack_place_experts (q computed when both are given)
 * Synchronizes (it checks slot_of first).  E_INVALID on null inputs or
 * outputs, E % P != 0, or a layer of slot_of that is not a permutation (then
 * nothing is written to q); E_UNSUPPORTED when 4 E bytes exceed the LDS. */
int routepack_project_demand(const routepack_problem *prob, const int64_t *agg, const int32_t *slot_of,
                             int64_t *rank_load, const int32_t *demand, int32_t *q, hipStream_t stream);

/* Row count and seed population (Sec. 3.2 and Alg. 2).
 * R_lb = max(1, min_rows, ceil(sum t / (C D)), ceil(#{t_i > C/2} / D));
 * R* = the first R >= R_lb for which FixedRowFFD with R*D cells succeeds
 * (the R*D longest samples by (-t, i) open the cells, every later one goes
 * to the lowest-index cell with room); certified = (R* == R_lb).  Seeds:
 * x_length (FFD), x_paired (EDPAwarePair of its cells, width 1, kept only if
 * strictly better), then n_trials - 2 randomized trials (WindowShuffle,
 * RandomizedBestFit, EDPAwarePair with width choice_width; Philox4x64-10
 * key (seed, 0), counter (draw, trial, phase, 3)); each in canonical form,
 * duplicates dropped, ordered by (score, discovery) and repeated cyclically
 * into pop_size members.
 *   lengths     int32 [N]            t_i in [1, C]
 *   q           int32 [N][L][P]      physical-rank demand
 *   r_star      [host] int32 out
 *   certified   [host] int32 out     1 when R* equals the lower bound
 *   population  int32 [pop_size][N]  out: canonical layouts
 *   scores      int64 [pop_size][3]  out
 *   info        [host] int32 [3] out or NULL: {R_lb, distinct seeds, trials kept}
 * Synchronizes.  E_INFEASIBLE, E_HEURISTIC, E_OVERFLOW as above;
 * E_UNSUPPORTED when L*P > 4096 or R*D > 4096. */
int routepack_pack_rows(const routepack_problem *prob, const int32_t *lengths, const int32_t *q,
                        uint64_t seed, int32_t n_trials, int32_t choice_width, int32_t pop_size,
                        int32_t *r_star, int32_t *certified, int32_t *population,
                        int64_t *scores, int32_t *info, hipStream_t stream);

/* Annealing schedule and proposal knobs (Sec. 4.1.2, Alg. 3). */
typedef struct routepack_anneal_params {
    int32_t n_sweeps;            /* temperature levels in this call, >= 0 */
    int32_t steps_per_sweep;     /* K proposal steps per member per level, >= 0 */
    const double *temperatures;  /* [host][n_sweeps] > 0, strictly decreasing */
    double t_next;               /* temperature of the level after this call (< last);
                                    <= 0 when this call ends the schedule (no resampling
                                    after its last level) */
    uint32_t p_guide_u32;        /* guided branch iff lo32(w0) < p_guide_u32 (0.8 -> 0xCCCCCCCD) */
    uint32_t rho_u32;            /* relocation iff hi32(w0) < rho_u32 (0.25 -> 0x40000000) */
    uint64_t seed;               /* Philox4x64-10 key (seed, 0) */
    int32_t sweep_offset;        /* global index of this call's first level */
    int32_t init_incumbent;      /* 1: x* := lowest-index argmin of the population */
    double *level_kernel_ms;     /* [host][n_sweeps] out or NULL: duration of each level's
                                    annealing kernel, from HIP events on `stream`; with
                                    ROUTEPACK_KERNEL_CHAIN_RUN (one kernel for all levels)
                                    every entry is that kernel's duration / n_sweeps */
    int32_t *level_kernel;       /* [host] out or NULL: the level kernel that ran
                                    (ROUTEPACK_KERNEL_*) */
} routepack_anneal_params;

/* Level kernels of routepack_anneal.  The library takes the first whose
 * shape limits the problem meets; the environment variable
 * ROUTEPACK_ANNEAL_KERNEL=chain_run|chain|wave|workgroup requests one (a request the
 * problem does not fit fails with ROUTEPACK_E_UNSUPPORTED).
 *   CHAIN_RUN  the CHAIN kernel for every level in one cooperative launch
 *              (member state stays on chip between levels; the level ends
 *              run in the same kernel): CHAIN shapes whose workgroups can
 *              all be resident at once
 *   CHAIN      one wave per member, lanes over (row-shard, layer) and cells:
 *              P in {4, 8, 16, 32, 64}, L <= 32 (L <= 64 when P >= 16),
 *              R G <= 128 (<= 64 when P >= 32), <= 16 slots per shard (<= 32
 *              when P = 64), N < 65536.  When the population cannot be
 *              resident at once and P = 32, the per-level launch may keep
 *              each member's cell array and the lengths in HBM to fit more
 *              members per CU (ROUTEPACK_CHAIN_LAYOUT=hbm asks for that
 *              layout, =lds forbids it); P = 64 always runs that layout, with
 *              the member pool, the cells' squared-length sums and the cost
 *              prefixes in HBM too (a 64-rank row is formed 16 ranks at a
 *              time), per level only
 *   WAVE       one wave per member, lanes over flat 64-entry strides:
 *              R G <= 512, member state within LDS
 *   WORKGROUP  one workgroup per member, state in HBM: every problem within
 *              the limits that routepack_anneal states */
#define ROUTEPACK_KERNEL_WORKGROUP 0
#define ROUTEPACK_KERNEL_WAVE 1
#define ROUTEPACK_KERNEL_CHAIN 2
#define ROUTEPACK_KERNEL_CHAIN_RUN 3

/* Fixed-row population annealing (Alg. 3) over n_sweeps levels.  Level n
 * (global index nn = sweep_offset + n) runs, for every member j independently,
 * K steps of: GuidedProposal (Sec. 4.1.2) with Philox words from counters
 * (k, nn, j, 0) and (k, nn, j, 1); a feasibility test (distinct cells,
 * capacity, no emptied cell) -- an infeasible proposal consumes the step;
 * IncrementalScore; the Metropolis test "s' < s lexicographically, or
 * u < exp(-max(Delta, 0) / T_n)" on the energy of Eq. pa-energy; and the
 * trajectory best (strict improvement).  After the level the incumbent x*
 * takes the lexicographic minimum of itself and every trajectory best
 * (strict, ascending j) and, unless the level is the schedule's last, the
 * terminal states are resampled systematically with Boltzmann weights for
 * the temperature change.  Moves never change R, coverage, capacity or the
 * shard topology.  Resuming with (population, x*, sweep_offset) is exact.
 *   lengths      int32 [N]
 *   q            int32 [N][L][P]
 *   n_rows       R (the fixed row count)
 *   population   int32 [pop_size][N]  in: start of level sweep_offset; out: start of
 *                the next level (resampled) or the terminal states (t_next <= 0)
 *   best_layout  int32 [N]    in/out x* (ignored on input when init_incumbent)
 *   best_score   int64 [3]    in/out Score(x*)
 *   trace        int64 [n_sweeps][pop_size][8] out or NULL: terminal score (3),
 *                trajectory-best score (3), accepted steps, evaluated steps
 *   parents      int32 [n_sweeps][pop_size] out or NULL: parent of each member
 *                after the level, -1 when no resampling followed it
 *   step_log     uint8 [n_sweeps][pop_size][K] out or NULL: 0 infeasible,
 *                1 rejected, 2 accepted
 * Synchronizes.  E_DEVICE on a HIP error, and when a grid barrier or a
 * hand-over wait of the whole-schedule kernel gives up: each wait polls a
 * shared error flag and gives up after 2^22 polls (ROUTEPACK_WAIT_SPINS in
 * the environment sets another bound, at least 32); every wave then leaves
 * the kernel and the outputs are undefined.  E_LAYOUT when a population
 * member (or the given x*) is not feasible for R or best_score does not
 * match x*; E_INTERNAL when the final
 * validation or the non-regression check fails; E_UNSUPPORTED (before any
 * device work) when P is not a power of two <= 64, L*P > 4096, R*G > 512,
 * G > 64, a shard holds more than 64 DP slots, or S > 4. */
int routepack_anneal(const routepack_problem *prob, const int32_t *lengths, const int32_t *q,
                     int32_t n_rows, int32_t pop_size, int32_t *population,
                     const routepack_anneal_params *params, int32_t *best_layout,
                     int64_t *best_score, int64_t *trace, int32_t *parents, uint8_t *step_log,
                     hipStream_t stream);

/* Exact objective of many layouts (Eqs. cell-token-statistics ..
 * lexicographic-score) with validation and the online load diagnostics of
 * Sec. 5.3 (Eqs. global-ep-cv and ep-efficiency).
 *   layouts    int32 [n_layouts][N]
 *   scores     int64 [n_layouts][3]  out (INT64_MAX x3 for an invalid layout)
 *   status     int32 [n_layouts]     out: 0, or bit 0 a cell id outside [0, R*D),
 *              bit 1 a cell over capacity, bit 2 an empty cell
 *   J          int64 [n_layouts][R*G] out or NULL: J per row-shard
 *   diag       double [n_layouts][8] out or NULL: CV_global (NaN without
 *              rank_load), S_EP, T_EP (raw tokens), eta_EP, sum A, max_g U,
 *              sum_g U (normalised by C), energy (Eq. pa-energy)
 *   rank_load  int64 [L][P] or NULL: window rank load for CV_global
 * Synchronizes (it sizes its scratch from a bound computed on the device).
 * E_OVERFLOW as above. */
int routepack_eval_objective(const routepack_problem *prob, const int32_t *lengths,
                             const int32_t *q, int32_t n_rows, int32_t n_layouts,
                             const int32_t *layouts, int64_t *scores, int32_t *status,
                             int64_t *J, double *diag, const int64_t *rank_load,
                             hipStream_t stream);

/* Lower bound on the row count (Sec. 3.2, Eqs. token-capacity and
 * min-row-count): R* from routepack_pack_rows is the minimum R_min whenever
 * it equals this bound, which can exceed the R_lb that pack_rows certifies
 * against.  K_bound, a lower bound on the cells of any layout, is the largest
 * of the token volume ceil(sum t / C), the cardinality bounds
 * ceil(#{t_i (k+1) > C} / k) for k >= 1 (no cell holds k + 1 samples longer
 * than C / (k + 1)), and Martello and Toth's L2 (1990) over every threshold
 * alpha in {0} and the lengths at most C / 2; R_bound = max(1, min_rows,
 * ceil(K_bound / D)).
 *   lengths     int32 [N] t_i in [1, C]
 *   r_bound     [host] int32 out
 *   cell_bound  [host] int64 out or NULL: K_bound
 * Synchronizes.  E_INFEASIBLE when some t_i is outside [1, C]. */
int routepack_row_lower_bound(const routepack_problem *prob, const int32_t *lengths, int32_t *r_bound,
                              int64_t *cell_bound, hipStream_t stream);

/* The fixed-bin feasibility check (Sec. 3.2, Eq. min-row-count): is there a
 * layout with R rows (Eqs. sample-bijection, nonempty-cell, token-capacity
 * with K = R D cells)?  Depth-first branch and bound in a fixed order, so the
 * verdict, the node count and the first solution are defined: samples in
 * (-t, i) order go to an open cell with room, lowest index first, then to
 * the first unopened cell; a sample as long as the previous one goes to no
 * lower cell; a branch is cut when fewer samples remain than unopened cells;
 * a node is one placement.  Run it for R from routepack_row_lower_bound up
 * to R* - 1: the first R found feasible is R_min, and if every one is
 * infeasible, R* is.
 *   n_rows       R
 *   node_budget  placements allowed (>= 0)
 *   status       [host] int32 out: 1 feasible, 0 infeasible, 2 unknown
 *                (budget spent)
 *   nodes        [host] int64 out or NULL: placements made
 *   layout       int32 [N] out or NULL: the cell of each sample in the
 *                first solution (written only when feasible)
 * Synchronizes.  A sample over capacity, or more cells than samples, is
 * infeasible (status 0, no node).  E_UNSUPPORTED when 8 R D + 4 N bytes
 * exceed 150 KiB of LDS. */
int routepack_fixed_bin_search(const routepack_problem *prob, const int32_t *lengths, int32_t n_rows,
                               int64_t node_budget, int32_t *status, int64_t *nodes, int32_t *layout,
                               hipStream_t stream);

/* QualityDiversitySelect (Sec. 4.1.1, diverse fixed-row seeding; Alg. 2, the
 * selection before the cyclic fill): the order in which canonical-distinct
 * candidate layouts enter the seed population.  Starting from candidate 0
 * (the exact-score winner), each step adds the candidate with the largest
 * min over chosen y of d(x, y) minus the primary-score gap
 * (s0(x) - s0(x_0)) / s0(x_0), the lower index on a tie, where
 * d = (A / N + B / N + E / (8 R 2^20)) / 3: A and B count the samples whose
 * cell, resp. row, holds a different sample set, and E is the L1 distance of
 * the row-feature sketches -- the 2 + L row features (token sum over D C,
 * sum of squared lengths over D C^2, and per layer sum_g max_p W over k D C,
 * floored in 20-bit fixed point) projected on 8 sign vectors (the bits of
 * Philox4x64-10 blocks (k, 0, 0, 4) under key (seed, 0)) and sorted over
 * the rows.  All arithmetic is integer, so the order is exact.
 *   candidates  int32 [n_cand][N]: layouts for R rows in (score, discovery)
 *               order, 1 <= n_cand <= 64
 *   primary     int64 [n_cand]: s0 of each candidate
 *   order       int32 [n_cand] out: the selection order (order[0] = 0)
 *   population  int32 [pop_size][N] out or NULL when pop_size = 0: the
 *               candidates in that order, repeated
 * Synchronizes.  E_LAYOUT when a candidate holds an id outside [0, R D), an
 * empty cell or a cell over capacity; E_UNSUPPORTED when N or R D exceeds
 * 65535, R exceeds 4096 or L exceeds 254; E_OVERFLOW when D C^2 >= 2^62. */
int routepack_select_population(const routepack_problem *prob, const int32_t *lengths,
                                const int32_t *q, int32_t n_rows, int32_t n_cand,
                                const int32_t *candidates, const int64_t *primary, uint64_t seed,
                                int32_t pop_size, int32_t *order, int32_t *population,
                                hipStream_t stream);

/* Human-readable name of a status code. */
const char *routepack_strerror(int code);

#ifdef __cplusplus
}
#endif
#endif /* ROUTEPACK_H */
