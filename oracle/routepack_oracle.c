/*
 * RoutePack planner hot path -- CPU ORACLE (test infrastructure only).
 *
 * This file is a plain, slow, obviously-correct C rendering of what the
 * planner computes (arXiv 2608.12146).  It exists to check the HIP path and
 * is never linked into it: only the tests, the smoke check and the CPU
 * baseline leg of the benchmark load it.  It shares no header, helper or
 * constant table with the HIP sources.
 *
 * Coverage and pins (tests/test_oracle_pins.py and
 * tests/test_oracle_operator_pins.py):
 *   or_philox4x64      Philox4x64-10 (Salmon et al., SC'11) -- pinned to
 *                      numpy.random.Philox.
 *   or_exp_det         exp(x) for x <= 0 by Cody-Waite reduction and a
 *                      degree-13 Taylor polynomial -- pinned by an error bound
 *                      against math.exp.
 *   or_aggregate       window aggregate L_{l,e} (Sec. 3.3) -- pinned to
 *                      numpy.sum.
 *   or_place           layer-local LPT (Alg. 1) -- pinned by hand-traced
 *                      cases, the Fig. 3 instance and invariants.
 *   or_project         physical-rank demand (Eq. physical-rank-demand) --
 *                      pinned to a one-hot einsum and the top-k invariant.
 *   or_score           Eqs. cell-token-statistics .. lexicographic-score in
 *                      fixed point -- pinned to exact rational brute force.
 *                      Its load diagnostics (Sec. 5.3, Eqs. global-ep-cv and
 *                      ep-efficiency) are pinned to the Fig. 3 numbers and to
 *                      numpy on random loads.
 *   or_pack_rows       R* search, FixedRowFFD and Alg. 2 seeding -- pinned by
 *                      invariants and exhaustive minimum row counts; its
 *                      operators (WindowShuffle, RandomizedBestFit,
 *                      EDPAwarePair; exported one at a time as or_seed_trial
 *                      and or_edp_pair) by hand-traced instances and by the
 *                      bounded draws of numpy's Philox.
 *   or_anneal          Alg. 3 population annealing -- incremental score pinned
 *                      to full rescoring at every step; GuidedProposal's
 *                      three roulettes and the random branch by one-step
 *                      proposals predicted from numpy's Philox and exact
 *                      row-shard costs; Eq. pa-energy and the normalised
 *                      Delta by accept thresholds at a known u; the strict
 *                      tie rules of the trajectory best and the incumbent by
 *                      equal-score twins.  The trajectory as a whole is
 *                      parity unpinned by the paper (special cases only:
 *                      all-tie acceptance, greedy limit, non-regression,
 *                      exhaustive optimum as a lower bound).
 *   or_resample(_at)   systematic resampling -- pinned by offspring counts,
 *                      the literal F_j >= u_m boundary at u_0 = 0, and exact
 *                      systematic resampling on real weights.  The 2^40 scale
 *                      at which weights are quantised is a determinism
 *                      constant, not a quantity of the paper: parity unpinned.
 *
 * Fixed-point convention: every cost is an int64 in units of 2^-F raw tokens,
 * so a normalised cost of the paper (divided by C) is value / (2^F * C).
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -pthread -shared.
 */
#define _GNU_SOURCE
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>


typedef struct {
    int32_t n_samples, n_layers, n_experts, top_k, n_ranks, n_dp, n_edp;
    const int32_t *dp_to_edp; /* [D] */
    int64_t capacity;
    int32_t n_stages;
    const int64_t *alpha_fp, *beta_fp; /* [S] */
    int32_t frac_bits;
    int32_t min_rows;
} or_problem;

enum { OR_OK = 0, OR_INVALID = -1, OR_INFEASIBLE = -2, OR_HEURISTIC = -3,
       OR_LAYOUT = -4, OR_OVERFLOW = -5, OR_INTERNAL = -7 };

/* ------------------------------------------------------------------------ */
/* Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11, "Parallel random numbers:
 * as easy as 1, 2, 3").  Ten rounds; each round multiplies counter words 0 and
 * 2 by the two round multipliers into 128-bit products, mixes the high halves
 * with the other counter words and the key, and the key is advanced by the
 * two Weyl constants between rounds. */
static const uint64_t PHILOX_M0 = 0xD2E7470EE14C6C93ULL;
static const uint64_t PHILOX_M1 = 0xCA5A826395121157ULL;
static const uint64_t PHILOX_W0 = 0x9E3779B97F4A7C15ULL;
static const uint64_t PHILOX_W1 = 0xBB67AE8584CAA73BULL;

void or_philox4x64(const uint64_t ctr_in[4], const uint64_t key_in[2], uint64_t out[4])
{
    uint64_t c[4] = {ctr_in[0], ctr_in[1], ctr_in[2], ctr_in[3]};
    uint64_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) { k0 += PHILOX_W0; k1 += PHILOX_W1; }
        unsigned __int128 p0 = (unsigned __int128)PHILOX_M0 * c[0];
        unsigned __int128 p1 = (unsigned __int128)PHILOX_M1 * c[2];
        uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
        uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
        uint64_t n0 = hi1 ^ c[1] ^ k0;
        uint64_t n1 = lo1;
        uint64_t n2 = hi0 ^ c[3] ^ k1;
        uint64_t n3 = lo0;
        c[0] = n0; c[1] = n1; c[2] = n2; c[3] = n3;
    }
    out[0] = c[0]; out[1] = c[1]; out[2] = c[2]; out[3] = c[3];
}

/* Bounded draw: floor(w * m / 2^64) (Lemire's multiply-shift). */
static uint64_t bnd(uint64_t w, uint64_t m)
{
    return (uint64_t)(((unsigned __int128)w * m) >> 64);
}

/* ------------------------------------------------------------------------ */
/* exp(x) for x <= 0, deterministic: Cody & Waite (1980) reduction
 * x = k ln2 + r with ln2 split into a 32-significant-bit head and a tail, then
 * the Taylor sum of e^r to degree 13 in Horner form with each coefficient the
 * double nearest 1/m!, then scaling by 2^k.  Every step is one IEEE operation;
 * the file is built without contraction. */
double or_exp_det(double x)
{
    const double INV_LN2 = 1.44269504088896338700e+00;
    const double LN2_HI = 6.93147180369123816490e-01; /* 32 significant bits */
    const double LN2_LO = 1.90821492927058770002e-10;
    if (!(x >= -708.0)) return 0.0;
    if (x > 0.0) x = 0.0;
    double kf = rint(x * INV_LN2);
    double r = (x - kf * LN2_HI) - kf * LN2_LO;
    double p = 1.0 / 6227020800.0;             /* 1/13! */
    p = p * r + 1.0 / 479001600.0;             /* 1/12! */
    p = p * r + 1.0 / 39916800.0;              /* 1/11! */
    p = p * r + 1.0 / 3628800.0;               /* 1/10! */
    p = p * r + 1.0 / 362880.0;                /* 1/9!  */
    p = p * r + 1.0 / 40320.0;                 /* 1/8!  */
    p = p * r + 1.0 / 5040.0;                  /* 1/7!  */
    p = p * r + 1.0 / 720.0;                   /* 1/6!  */
    p = p * r + 1.0 / 120.0;                   /* 1/5!  */
    p = p * r + 1.0 / 24.0;                    /* 1/4!  */
    p = p * r + 1.0 / 6.0;                     /* 1/3!  */
    p = p * r + 0.5;                           /* 1/2!  */
    p = p * r + 1.0;                           /* 1/1!  */
    p = p * r + 1.0;                           /* 1/0!  */
    return ldexp(p, (int)kf);
}

/* ------------------------------------------------------------------------ */
/* Window aggregate: L_{l,e} = sum_i a_{i,l,e} (Sec. 3.3, Layer-wise expert
 * placement), accumulated in int64. */
void or_aggregate(int32_t N, int32_t L, int32_t E, const int32_t *demand, int64_t *agg)
{
    for (int64_t x = 0; x < (int64_t)L * E; ++x) agg[x] = 0;
    for (int64_t i = 0; i < N; ++i)
        for (int64_t l = 0; l < L; ++l)
            for (int64_t e = 0; e < E; ++e)
                agg[l * E + e] += demand[(i * L + l) * E + e];
}

/* Layer-local LPT placement (Alg. 1).  Experts of a layer are visited by
 * (-L_{l,e}, e); each goes to the least-loaded rank by (G_p, p) among ranks
 * with fewer than H experts and takes that rank's next slot p*H + n_p.
 * slot_of[l][e] = pi_l(e); owner(v) = v / H; rank_load[l][p] = G_{l,p}. */
static const int64_t *g_sort_keys;
static int cmp_lpt(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    int64_t kx = g_sort_keys[x], ky = g_sort_keys[y];
    if (kx != ky) return kx > ky ? -1 : 1; /* larger load first */
    return x < y ? -1 : (x > y);
}

int or_place(int32_t L, int32_t E, int32_t P, const int64_t *agg, int32_t *slot_of,
             int64_t *rank_load)
{
    if (P <= 0 || E % P != 0) return OR_INVALID;
    int32_t H = E / P;
    int32_t *order = malloc(sizeof(int32_t) * (E > 0 ? E : 1));
    int32_t *nfill = malloc(sizeof(int32_t) * P);
    for (int32_t l = 0; l < L; ++l) {
        const int64_t *Ll = agg + (int64_t)l * E;
        int64_t *G = rank_load + (int64_t)l * P;
        for (int32_t p = 0; p < P; ++p) { G[p] = 0; nfill[p] = 0; }
        for (int32_t e = 0; e < E; ++e) order[e] = e;
        g_sort_keys = Ll;
        qsort(order, E, sizeof(int32_t), cmp_lpt);
        for (int32_t k = 0; k < E; ++k) {
            int32_t e = order[k];
            int32_t best = -1;
            for (int32_t p = 0; p < P; ++p) {
                if (nfill[p] >= H) continue;
                if (best < 0 || G[p] < G[best]) best = p; /* ties keep lower p */
            }
            slot_of[(int64_t)l * E + e] = best * H + nfill[best];
            G[best] += Ll[e];
            nfill[best] += 1;
        }
    }
    free(order); free(nfill);
    return OR_OK;
}

/* Physical-rank demand q_{i,l,p} = sum over e with owner(pi_l(e)) = p of
 * a_{i,l,e} (Eq. physical-rank-demand). */
int or_project(int32_t N, int32_t L, int32_t E, int32_t P, const int32_t *demand,
               const int32_t *slot_of, int32_t *q)
{
    if (P <= 0 || E % P != 0) return OR_INVALID;
    int32_t H = E / P;
    for (int64_t x = 0; x < (int64_t)N * L * P; ++x) q[x] = 0;
    for (int64_t i = 0; i < N; ++i)
        for (int64_t l = 0; l < L; ++l)
            for (int64_t e = 0; e < E; ++e) {
                int32_t p = slot_of[l * E + e] / H;
                q[(i * L + l) * P + p] += demand[(i * L + l) * E + e];
            }
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Topology helpers: slots of shard g in ascending order. */
typedef struct {
    int32_t G, D;
    int32_t *count;   /* [G] */
    int32_t *slots;   /* [G][D] ascending slots of each shard */
} topo_t;

static int topo_build(const or_problem *pb, topo_t *tp)
{
    tp->G = pb->n_edp; tp->D = pb->n_dp;
    if (tp->G <= 0 || tp->D <= 0 || tp->G > tp->D) return OR_INVALID;
    tp->count = calloc(tp->G, sizeof(int32_t));
    tp->slots = calloc((size_t)tp->G * tp->D, sizeof(int32_t));
    for (int32_t d = 0; d < tp->D; ++d) {
        int32_t g = pb->dp_to_edp[d];
        if (g < 0 || g >= tp->G) return OR_INVALID;
        tp->slots[(int64_t)g * tp->D + tp->count[g]++] = d;
    }
    for (int32_t g = 0; g < tp->G; ++g) if (tp->count[g] == 0) return OR_INVALID;
    return OR_OK;
}
static void topo_free(topo_t *tp) { free(tp->count); free(tp->slots); }

/* ------------------------------------------------------------------------ */
/* Exact score of a layout (Eqs. cell-token-statistics, stage-aware-attention,
 * row-expert-load, row-expert-cost, lexicographic-score), multiplied by the
 * positive constant 2^F * C so that every term is an integer:
 *   cost_s(c) = alpha_s * T_c + beta_s * Q2_c       (T = sum t, Q2 = sum t^2)
 *   A(r,g)    = sum_s max_{d in D_g} cost_s(r*D+d)
 *   W(r,g,l,p)= sum_{d in D_g} sum_{i in cell(r,d)} q[i][l][p]
 *   E(r,g)    = 2^F * sum_l max_p W(r,g,l,p)
 *   J = A + E; U_g = sum_r J(r,g); s = (max_g U, sum_g U, max_{r,g} J).
 * layout[i] = cell id r*D + d.  Returns a status bitmask: bit 0 a cell id out
 * of range, bit 1 a cell over capacity, bit 2 an empty cell; on a nonzero
 * status the score is set to INT64_MAX. */
int or_score(const or_problem *pb, const int32_t *t, const int32_t *q, int32_t R,
             const int32_t *layout, int64_t *score, int64_t *J_out, double *diag,
             const int64_t *rank_load)
{
    topo_t tp;
    if (topo_build(pb, &tp) != OR_OK) return -1;
    int32_t N = pb->n_samples, L = pb->n_layers, P = pb->n_ranks, D = pb->n_dp, G = pb->n_edp;
    int32_t S = pb->n_stages;
    int64_t B = (int64_t)R * D;
    int64_t C = pb->capacity;
    int status = 0;
    int64_t *T = calloc(B > 0 ? B : 1, sizeof(int64_t));
    int64_t *Q2 = calloc(B > 0 ? B : 1, sizeof(int64_t));
    int64_t *cnt = calloc(B > 0 ? B : 1, sizeof(int64_t));
    int64_t *W = calloc((size_t)R * G * L * P + 1, sizeof(int64_t));
    int64_t *J = calloc((size_t)R * G + 1, sizeof(int64_t));
    int64_t *A = calloc((size_t)R * G + 1, sizeof(int64_t));
    for (int32_t i = 0; i < N; ++i) {
        int32_t c = layout[i];
        if (c < 0 || c >= B) { status |= 1; continue; }
        T[c] += t[i];
        Q2[c] += (int64_t)t[i] * t[i];
        cnt[c] += 1;
        int32_t r = c / D, d = c % D, g = pb->dp_to_edp[d];
        int64_t *w = W + ((int64_t)r * G + g) * L * P;
        for (int64_t x = 0; x < (int64_t)L * P; ++x) w[x] += q[(int64_t)i * L * P + x];
    }
    for (int64_t c = 0; c < B; ++c) {
        if (T[c] > C) status |= 2;
        if (cnt[c] == 0) status |= 4;
    }
    if (status) {
        score[0] = score[1] = score[2] = INT64_MAX;
        if (J_out) for (int64_t h = 0; h < (int64_t)R * G; ++h) J_out[h] = INT64_MAX;
        if (diag) for (int k = 0; k < 8; ++k) diag[k] = NAN;
        goto done;
    }
    for (int32_t r = 0; r < R; ++r)
        for (int32_t g = 0; g < G; ++g) {
            int64_t a = 0;
            for (int32_t s = 0; s < S; ++s) {
                int64_t mx = 0;
                for (int32_t k = 0; k < tp.count[g]; ++k) {
                    int64_t c = (int64_t)r * D + tp.slots[(int64_t)g * D + k];
                    int64_t cost = pb->alpha_fp[s] * T[c] + pb->beta_fp[s] * Q2[c];
                    if (k == 0 || cost > mx) mx = cost;
                }
                a += mx;
            }
            const int64_t *w = W + ((int64_t)r * G + g) * L * P;
            int64_t esum = 0;
            for (int32_t l = 0; l < L; ++l) {
                int64_t mx = w[(int64_t)l * P];
                for (int32_t p = 1; p < P; ++p) if (w[(int64_t)l * P + p] > mx) mx = w[(int64_t)l * P + p];
                esum += mx;
            }
            A[(int64_t)r * G + g] = a;
            J[(int64_t)r * G + g] = a + (esum << pb->frac_bits);
        }
    {
        int64_t s0 = 0, s1 = 0, s2 = 0;
        for (int32_t g = 0; g < G; ++g) {
            int64_t U = 0;
            for (int32_t r = 0; r < R; ++r) U += J[(int64_t)r * G + g];
            if (g == 0 || U > s0) s0 = U;
            s1 += U;
        }
        for (int64_t h = 0; h < (int64_t)R * G; ++h) if (h == 0 || J[h] > s2) s2 = J[h];
        score[0] = s0; score[1] = s1; score[2] = s2;
        if (J_out) memcpy(J_out, J, sizeof(int64_t) * R * G);
    }
    if (diag) {
        /* Online load diagnostics, raw tokens for W, normalised costs. */
        double scale = (double)((int64_t)1 << pb->frac_bits) * (double)C;
        double cv = NAN;
        if (rank_load) {
            cv = 0.0;
            for (int32_t l = 0; l < L; ++l) {
                double mean = 0.0;
                for (int32_t p = 0; p < P; ++p) mean += (double)rank_load[(int64_t)l * P + p];
                mean /= (double)P;
                double var = 0.0;
                for (int32_t p = 0; p < P; ++p) {
                    double dv = (double)rank_load[(int64_t)l * P + p] - mean;
                    var += dv * dv;
                }
                var /= (double)P;
                cv += mean > 0.0 ? sqrt(var) / mean : 0.0;
            }
            cv = L > 0 ? cv / (double)L : 0.0;
        }
        double s_ep = 0.0, t_ep = 0.0, ideal = 0.0, att = 0.0;
        for (int32_t r = 0; r < R; ++r)
            for (int32_t l = 0; l < L; ++l) {
                int64_t mx = 0; double best_mean = 0.0;
                for (int32_t g = 0; g < G; ++g) {
                    const int64_t *w = W + (((int64_t)r * G + g) * L + l) * P;
                    int64_t tot = 0;
                    for (int32_t p = 0; p < P; ++p) { if (w[p] > mx) mx = w[p]; tot += w[p]; }
                    double mean = (double)tot / (double)P;
                    if (mean > best_mean) best_mean = mean;
                }
                s_ep += (double)mx;
                if ((double)mx > t_ep) t_ep = (double)mx;
                ideal += best_mean;
            }
        for (int64_t h = 0; h < (int64_t)R * G; ++h) att += (double)A[h] / scale;
        double S0 = (double)score[0] / scale, S1 = (double)score[1] / scale, S2 = (double)score[2] / scale;
        diag[0] = cv;
        diag[1] = s_ep;
        diag[2] = t_ep;
        diag[3] = s_ep > 0.0 ? ideal / s_ep : 1.0;
        diag[4] = att;
        diag[5] = S0;
        diag[6] = S1;
        diag[7] = (S0 + 1e-6 * S1) + 1e-9 * S2;
    }
done:
    free(T); free(Q2); free(cnt); free(W); free(J); free(A);
    topo_free(&tp);
    return status;
}

/* ------------------------------------------------------------------------ */
/* Bound check.  Every W entry of a capacity-feasible layout is at most
 * Wb = min(max_l sum_{i,p} q[i][l][p], rate * maxD * C), where rate =
 * max_i ceil(max_{l,p} q[i][l][p] / t_i) and maxD is the largest shard: the
 * samples of one row-shard hold at most maxD * C tokens.  Then every J is at
 * most Ab + Eb with Ab = sum_s (alpha_s C + beta_s C^2), Eb = 2^F L Wb, and
 * R*G*(Ab+Eb+1) must stay below 2^53 so every score component is exact in
 * int64 and in a double. */
static int overflow_check(const or_problem *pb, const int32_t *t, const int32_t *q, int32_t R,
                          int64_t *wb_out)
{
    int32_t N = pb->n_samples, L = pb->n_layers, P = pb->n_ranks;
    long double lim = 9007199254740992.0L; /* 2^53 */
    int64_t wb = 0, rate = 0;
    for (int32_t l = 0; l < L; ++l) {
        int64_t tot = 0;
        for (int32_t i = 0; i < N; ++i)
            for (int32_t p = 0; p < P; ++p) tot += q[((int64_t)i * L + l) * P + p];
        if (tot > wb) wb = tot;
    }
    for (int32_t i = 0; i < N; ++i) {
        int64_t mx = 0;
        for (int64_t x = 0; x < (int64_t)L * P; ++x)
            if (q[(int64_t)i * L * P + x] > mx) mx = q[(int64_t)i * L * P + x];
        int64_t r = t[i] > 0 ? (mx + t[i] - 1) / t[i] : mx;
        if (r > rate) rate = r;
    }
    int32_t maxd = 0;
    {
        int32_t *cnt = calloc(pb->n_edp, sizeof(int32_t));
        for (int32_t d = 0; d < pb->n_dp; ++d) cnt[pb->dp_to_edp[d]]++;
        for (int32_t g = 0; g < pb->n_edp; ++g) if (cnt[g] > maxd) maxd = cnt[g];
        free(cnt);
    }
    long double wcap = (long double)rate * maxd * (long double)pb->capacity;
    if (wcap < (long double)wb) wb = (int64_t)wcap;
    long double C = (long double)pb->capacity;
    long double ab = 0.0L;
    for (int32_t s = 0; s < pb->n_stages; ++s)
        ab += (long double)pb->alpha_fp[s] * C + (long double)pb->beta_fp[s] * C * C;
    long double eb = ldexpl((long double)L * (long double)wb, pb->frac_bits);
    long double tot = (long double)R * pb->n_edp * (ab + eb + 1.0L);
    if (wb_out) *wb_out = wb;
    if (!(tot < lim)) return OR_OVERFLOW;
    if (!(ldexpl((long double)pb->capacity, pb->frac_bits) < lim)) return OR_OVERFLOW;
    return OR_OK;
}

static int check_problem(const or_problem *pb)
{
    if (pb->n_samples < 0 || pb->n_layers < 0 || pb->n_experts < 0 || pb->n_ranks <= 0) return OR_INVALID;
    if (pb->n_experts % pb->n_ranks != 0) return OR_INVALID;
    if (pb->n_dp <= 0 || pb->n_edp <= 0 || pb->capacity <= 0 || pb->n_stages < 1) return OR_INVALID;
    if (pb->frac_bits < 0 || pb->frac_bits > 30) return OR_INVALID;
    for (int32_t s = 0; s < pb->n_stages; ++s)
        if (pb->alpha_fp[s] < 0 || pb->beta_fp[s] < 0) return OR_INVALID;
    topo_t tp;
    int rc = topo_build(pb, &tp);
    topo_free(&tp);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Fixed-row packing: row-count search, FixedRowFFD, and Alg. 2 seeding. */

static const int32_t *g_len;
static int cmp_len_desc(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    if (g_len[x] != g_len[y]) return g_len[x] > g_len[y] ? -1 : 1;
    return x < y ? -1 : (x > y);
}

/* FixedRowFFD with K cells: the K longest samples (by (-t, i)) open the cells
 * in order; each later sample goes to the lowest-index cell with room.
 * Returns 1 on success and fills cell_of. */
static int fixed_row_ffd(int32_t N, const int32_t *t, int64_t C, int64_t K,
                         const int32_t *sigma, int32_t *cell_of)
{
    if (K > N || K <= 0) return 0;
    int64_t *T = calloc(K, sizeof(int64_t));
    int ok = 1;
    for (int64_t h = 0; h < N; ++h) {
        int32_t i = sigma[h];
        if (h < K) { cell_of[i] = (int32_t)h; T[h] = t[i]; continue; }
        int64_t c;
        for (c = 0; c < K; ++c) if (T[c] + t[i] <= C) break;
        if (c == K) { ok = 0; break; }
        cell_of[i] = (int32_t)c;
        T[c] += t[i];
    }
    free(T);
    return ok;
}

/* One uint64 word for seed construction: word 0 of the Philox block with key
 * (seed, 0) and counter (draw, trial, phase, 3). */
static uint64_t seed_word(uint64_t seed, uint64_t draw, uint64_t trial, uint64_t phase)
{
    uint64_t ctr[4] = {draw, trial, phase, 3}, key[2] = {seed, 0}, out[4];
    or_philox4x64(ctr, key, out);
    return out[0];
}

typedef struct { int64_t inc, pk; int32_t h; } pair_cand;
static int cmp_pair_cand(const void *a, const void *b)
{
    const pair_cand *x = a, *y = b;
    if (x->inc != y->inc) return x->inc < y->inc ? -1 : 1;
    if (x->pk != y->pk) return x->pk < y->pk ? -1 : 1;
    return x->h < y->h ? -1 : (x->h > y->h);
}
typedef struct { int64_t peak; int32_t k; } peak_key;
static int cmp_peak(const void *a, const void *b)
{
    const peak_key *x = a, *y = b;
    if (x->peak != y->peak) return x->peak > y->peak ? -1 : 1;
    return x->k < y->k ? -1 : (x->k > y->k);
}

/* EDPAwarePair (Sec. 4.1.1): completed cells (cellk[i] = k in [0,K)) are
 * visited by decreasing routed peak sum_l max_p Q_k[l][p] (ties by k) and each
 * is inserted into a row-shard (r,g) that still has an empty slot, ranked by
 * (increase of sum_l max_p W(r,g), resulting max_{l,p} W(r,g), r, g); the rank
 * is drawn among the leading w' = min(w, #candidates) with weight
 * 2^(w'-1-rank); the cell takes the lowest empty slot of D_g. */
static void edp_aware_pair(const or_problem *pb, const topo_t *tp, const int32_t *q,
                           int32_t R, const int32_t *cellk, int32_t w, uint64_t seed,
                           uint64_t trial, int32_t *out_layout)
{
    int32_t N = pb->n_samples, L = pb->n_layers, P = pb->n_ranks, D = pb->n_dp, G = pb->n_edp;
    int64_t K = (int64_t)R * D, LP = (int64_t)L * P, RG = (int64_t)R * G;
    int64_t *Q = calloc((size_t)K * LP + 1, sizeof(int64_t));
    for (int32_t i = 0; i < N; ++i)
        for (int64_t x = 0; x < LP; ++x) Q[cellk[i] * LP + x] += q[(int64_t)i * LP + x];
    peak_key *order = malloc(sizeof(peak_key) * K);
    for (int64_t k = 0; k < K; ++k) {
        int64_t pk = 0;
        for (int32_t l = 0; l < L; ++l) {
            int64_t mx = Q[k * LP + (int64_t)l * P];
            for (int32_t p = 1; p < P; ++p) if (Q[k * LP + (int64_t)l * P + p] > mx) mx = Q[k * LP + (int64_t)l * P + p];
            pk += mx;
        }
        order[k].peak = pk; order[k].k = (int32_t)k;
    }
    qsort(order, K, sizeof(peak_key), cmp_peak);
    int64_t *W = calloc((size_t)RG * LP + 1, sizeof(int64_t));
    int32_t *filled = calloc(RG, sizeof(int32_t));
    int32_t *cell_to = malloc(sizeof(int32_t) * K);
    pair_cand *cand = malloc(sizeof(pair_cand) * RG);
    for (int64_t pos = 0; pos < K; ++pos) {
        int32_t k = order[pos].k;
        int32_t nc = 0;
        for (int64_t h = 0; h < RG; ++h) {
            int32_t g = (int32_t)(h % G);
            if (filled[h] >= tp->count[g]) continue;
            int64_t before = 0, after = 0, pkmax = 0;
            for (int32_t l = 0; l < L; ++l) {
                int64_t mb = 0, ma = 0;
                for (int32_t p = 0; p < P; ++p) {
                    int64_t wv = W[h * LP + (int64_t)l * P + p];
                    int64_t av = wv + Q[(int64_t)k * LP + (int64_t)l * P + p];
                    if (p == 0 || wv > mb) mb = wv;
                    if (p == 0 || av > ma) ma = av;
                }
                before += mb; after += ma;
                if (ma > pkmax) pkmax = ma;
            }
            cand[nc].inc = after - before; cand[nc].pk = pkmax; cand[nc].h = (int32_t)h;
            ++nc;
        }
        qsort(cand, nc, sizeof(pair_cand), cmp_pair_cand);
        int32_t wp = w < nc ? w : nc;
        int32_t rho = 0;
        if (wp > 1) {
            uint64_t total = (((uint64_t)1) << wp) - 1;
            uint64_t pick = bnd(seed_word(seed, (uint64_t)pos, trial, 2), total);
            uint64_t pref = 0;
            for (rho = 0; rho < wp; ++rho) {
                pref += ((uint64_t)1) << (wp - 1 - rho);
                if (pref > pick) break;
            }
        }
        int32_t h = cand[rho].h;
        int32_t r = h / G, g = h % G;
        int32_t d = tp->slots[(int64_t)g * D + filled[h]];
        filled[h] += 1;
        for (int64_t x = 0; x < LP; ++x) W[h * LP + x] += Q[(int64_t)k * LP + x];
        cell_to[k] = r * D + d;
    }
    for (int32_t i = 0; i < N; ++i) out_layout[i] = cell_to[cellk[i]];
    free(Q); free(order); free(W); free(filled); free(cell_to); free(cand);
}

/* Canonicalize (Sec. 4.1.1): sample ids sorted within each cell; within each
 * row-shard the cells are ordered by their sorted id tuples and given the
 * shard's slots in ascending order; rows are ordered by their tuple of cell
 * tuples (slots 0..D-1). */
typedef struct { int32_t *ids; int32_t n; } tuple_t;
static int tuple_cmp(const tuple_t *a, const tuple_t *b)
{
    int32_t m = a->n < b->n ? a->n : b->n;
    for (int32_t k = 0; k < m; ++k)
        if (a->ids[k] != b->ids[k]) return a->ids[k] < b->ids[k] ? -1 : 1;
    return a->n < b->n ? -1 : (a->n > b->n);
}
static int cmp_int32(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return x < y ? -1 : (x > y);
}
static tuple_t *g_cells;
static int32_t g_D;
static int cmp_cell_idx(const void *a, const void *b)
{
    return tuple_cmp(&g_cells[*(const int32_t *)a], &g_cells[*(const int32_t *)b]);
}
static int cmp_row_idx(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    for (int32_t d = 0; d < g_D; ++d) {
        int c = tuple_cmp(&g_cells[(int64_t)x * g_D + d], &g_cells[(int64_t)y * g_D + d]);
        if (c) return c;
    }
    return 0;
}

static void canonical_layout(const or_problem *pb, const topo_t *tp, int32_t R,
                         const int32_t *layout, int32_t *out)
{
    int32_t N = pb->n_samples, D = pb->n_dp, G = pb->n_edp;
    int64_t B = (int64_t)R * D;
    tuple_t *cells = calloc(B, sizeof(tuple_t));
    for (int32_t i = 0; i < N; ++i) cells[layout[i]].n++;
    for (int64_t c = 0; c < B; ++c) { cells[c].ids = malloc(sizeof(int32_t) * (cells[c].n + 1)); cells[c].n = 0; }
    for (int32_t i = 0; i < N; ++i) { tuple_t *tc = &cells[layout[i]]; tc->ids[tc->n++] = i; }
    for (int64_t c = 0; c < B; ++c) qsort(cells[c].ids, cells[c].n, sizeof(int32_t), cmp_int32);
    /* Step 1: within each (r, g), order the shard's cells. */
    tuple_t *placed = calloc(B, sizeof(tuple_t));
    int32_t *idx = malloc(sizeof(int32_t) * D);
    for (int32_t r = 0; r < R; ++r)
        for (int32_t g = 0; g < G; ++g) {
            int32_t m = tp->count[g];
            for (int32_t k = 0; k < m; ++k) idx[k] = r * D + tp->slots[(int64_t)g * D + k];
            g_cells = cells;
            qsort(idx, m, sizeof(int32_t), cmp_cell_idx);
            for (int32_t k = 0; k < m; ++k)
                placed[(int64_t)r * D + tp->slots[(int64_t)g * D + k]] = cells[idx[k]];
        }
    /* Step 2: order the rows. */
    int32_t *rows = malloc(sizeof(int32_t) * (R > 0 ? R : 1));
    for (int32_t r = 0; r < R; ++r) rows[r] = r;
    g_cells = placed; g_D = D;
    qsort(rows, R, sizeof(int32_t), cmp_row_idx);
    for (int32_t nr = 0; nr < R; ++nr)
        for (int32_t d = 0; d < D; ++d) {
            tuple_t *tc = &placed[(int64_t)rows[nr] * D + d];
            for (int32_t k = 0; k < tc->n; ++k) out[tc->ids[k]] = nr * D + d;
        }
    for (int64_t c = 0; c < B; ++c) free(cells[c].ids);
    free(cells); free(placed); free(idx); free(rows);
}

typedef struct { int64_t T; int32_t n; int32_t c; } fit_key;
static int cmp_fit(const void *a, const void *b)
{
    const fit_key *x = a, *y = b;
    if (x->T != y->T) return x->T > y->T ? -1 : 1; /* decreasing occupancy */
    if (x->n != y->n) return x->n < y->n ? -1 : 1; /* then cardinality */
    return x->c < y->c ? -1 : (x->c > y->c);        /* then index */
}

/* One randomized seed trial (Alg. 2, loop body): WindowShuffle of the
 * (-t, i) order, the first K samples open cells, RandomizedBestFit for the
 * rest, then EDPAwarePair.  Returns 1 and fills layout on success. */
static int seed_trial(const or_problem *pb, const topo_t *tp, const int32_t *t, const int32_t *q,
                      int32_t R, const int32_t *sigma, int32_t w, uint64_t seed, uint64_t trial,
                      int32_t *layout, int32_t *pi_out, int32_t *cellk_out)
{
    int32_t N = pb->n_samples;
    int64_t K = (int64_t)R * pb->n_dp, C = pb->capacity;
    int32_t *remaining = malloc(sizeof(int32_t) * N);
    int32_t *pi = malloc(sizeof(int32_t) * N);
    memcpy(remaining, sigma, sizeof(int32_t) * N);
    int32_t nrem = N;
    for (int32_t h = 0; h < N; ++h) {
        int32_t wp = w < nrem ? w : nrem;
        int32_t pos = (int32_t)bnd(seed_word(seed, (uint64_t)h, trial, 0), (uint64_t)wp);
        pi[h] = remaining[pos];
        memmove(remaining + pos, remaining + pos + 1, sizeof(int32_t) * (nrem - pos - 1));
        nrem -= 1;
    }
    int32_t *cellk = malloc(sizeof(int32_t) * N);
    int64_t *T = calloc(K, sizeof(int64_t));
    int32_t *cnt = calloc(K, sizeof(int32_t));
    fit_key *feas = malloc(sizeof(fit_key) * K);
    int ok = 1;
    for (int32_t h = 0; h < N && ok; ++h) {
        int32_t i = pi[h];
        if (h < K) { cellk[i] = h; T[h] = t[i]; cnt[h] = 1; continue; }
        int32_t nf = 0;
        for (int64_t c = 0; c < K; ++c)
            if (T[c] + t[i] <= C) { feas[nf].T = T[c]; feas[nf].n = cnt[c]; feas[nf].c = (int32_t)c; ++nf; }
        if (nf == 0) { ok = 0; break; }
        qsort(feas, nf, sizeof(fit_key), cmp_fit);
        int32_t wp = w < nf ? w : nf;
        int32_t rho = (int32_t)bnd(seed_word(seed, (uint64_t)h, trial, 1), (uint64_t)wp);
        int32_t c = feas[rho].c;
        cellk[i] = c; T[c] += t[i]; cnt[c] += 1;
    }
    if (pi_out) memcpy(pi_out, pi, sizeof(int32_t) * N);
    if (ok && cellk_out) memcpy(cellk_out, cellk, sizeof(int32_t) * N);
    if (ok) edp_aware_pair(pb, tp, q, R, cellk, w, seed, trial, layout);
    free(remaining); free(pi); free(cellk); free(T); free(cnt); free(feas);
    return ok;
}

static int lex_lt(const int64_t *a, const int64_t *b)
{
    if (a[0] != b[0]) return a[0] < b[0];
    if (a[1] != b[1]) return a[1] < b[1];
    return a[2] < b[2];
}

typedef struct { int64_t s[3]; int32_t disc; } cand_key;
static int cmp_cand(const void *a, const void *b)
{
    const cand_key *x = a, *y = b;
    if (lex_lt(x->s, y->s)) return -1;
    if (lex_lt(y->s, x->s)) return 1;
    return x->disc < y->disc ? -1 : (x->disc > y->disc);
}

/* Row-count search and Alg. 2 seeding.  population[pop][N] receives the
 * canonical seeds ordered by (score, discovery order) and repeated
 * cyclically; scores[pop][3] their exact scores.  extra (may be NULL) gets
 * {R_lb, number of distinct seeds, number of successful trials}. */
int or_pack_rows(const or_problem *pb, const int32_t *t, const int32_t *q, uint64_t seed,
                 int32_t n_trials, int32_t w, int32_t pop, int32_t *r_star, int32_t *certified,
                 int32_t *population, int64_t *scores, int32_t *extra)
{
    int rc = check_problem(pb);
    if (rc) return rc;
    if (n_trials < 2 || w < 1 || pop < 1) return OR_INVALID;
    int32_t N = pb->n_samples, D = pb->n_dp;
    int64_t C = pb->capacity;
    if (N < 1) return OR_INVALID;
    int64_t sum_t = 0, big = 0, tmax = 0;
    for (int32_t i = 0; i < N; ++i) {
        if (t[i] < 1) return OR_INVALID;
        sum_t += t[i];
        if (t[i] > tmax) tmax = t[i];
        if (2 * (int64_t)t[i] > C) big += 1;
    }
    int64_t r_lb = 1;
    if (pb->min_rows > r_lb) r_lb = pb->min_rows;
    int64_t a = (sum_t + C * D - 1) / (C * D);
    if (a > r_lb) r_lb = a;
    int64_t b = (big + D - 1) / D;
    if (b > r_lb) r_lb = b;
    int64_t r_max = N / D;
    if (tmax > C || r_lb > r_max) return OR_INFEASIBLE;
    int32_t *sigma = malloc(sizeof(int32_t) * N);
    for (int32_t i = 0; i < N; ++i) sigma[i] = i;
    g_len = t;
    qsort(sigma, N, sizeof(int32_t), cmp_len_desc);
    int32_t *x_len = malloc(sizeof(int32_t) * N);
    int64_t R = -1;
    for (int64_t r = r_lb; r <= r_max; ++r)
        if (fixed_row_ffd(N, t, C, r * D, sigma, x_len)) { R = r; break; }
    if (R < 0) { free(sigma); free(x_len); return OR_HEURISTIC; }
    if ((rc = overflow_check(pb, t, q, (int32_t)R, NULL))) { free(sigma); free(x_len); return rc; }
    *r_star = (int32_t)R;
    *certified = (R == r_lb);
    topo_t tp;
    topo_build(pb, &tp);
    int32_t M = n_trials;
    int32_t *cand = malloc(sizeof(int32_t) * (size_t)M * N);   /* canonical layouts */
    cand_key *keys = malloc(sizeof(cand_key) * M);
    int32_t ncand = 0, n_ok_trials = 0;
    int32_t *tmp = malloc(sizeof(int32_t) * N), *tmp2 = malloc(sizeof(int32_t) * N);
    for (int32_t m = 0; m < M; ++m) {
        /* m = 0: x_length; m = 1: x_paired; m >= 2: trial m-1. */
        int ok = 1;
        if (m == 0) memcpy(tmp, x_len, sizeof(int32_t) * N);
        else if (m == 1) {
            int32_t *paired = malloc(sizeof(int32_t) * N);
            edp_aware_pair(pb, &tp, q, (int32_t)R, x_len, 1, seed, 0, paired);
            int64_t s_len[3], s_pair[3];
            or_score(pb, t, q, (int32_t)R, x_len, s_len, NULL, NULL, NULL);
            or_score(pb, t, q, (int32_t)R, paired, s_pair, NULL, NULL, NULL);
            memcpy(tmp, lex_lt(s_pair, s_len) ? paired : x_len, sizeof(int32_t) * N);
            free(paired);
        } else {
            ok = seed_trial(pb, &tp, t, q, (int32_t)R, sigma, w, seed, (uint64_t)(m - 1), tmp, NULL, NULL);
            if (ok) {
                int64_t s[3];
                if (or_score(pb, t, q, (int32_t)R, tmp, s, NULL, NULL, NULL) != 0) ok = 0;
            }
            if (ok) n_ok_trials++;
        }
        if (!ok) continue;
        canonical_layout(pb, &tp, (int32_t)R, tmp, tmp2);
        int dup = 0;
        for (int32_t c = 0; c < ncand && !dup; ++c)
            if (memcmp(cand + (size_t)c * N, tmp2, sizeof(int32_t) * N) == 0) dup = 1;
        if (dup) continue;
        memcpy(cand + (size_t)ncand * N, tmp2, sizeof(int32_t) * N);
        or_score(pb, t, q, (int32_t)R, tmp2, keys[ncand].s, NULL, NULL, NULL);
        keys[ncand].disc = ncand;
        ncand++;
    }
    qsort(keys, ncand, sizeof(cand_key), cmp_cand);
    for (int32_t m = 0; m < pop; ++m) {
        const cand_key *k = &keys[m % ncand];
        memcpy(population + (size_t)m * N, cand + (size_t)k->disc * N, sizeof(int32_t) * N);
        memcpy(scores + (size_t)m * 3, k->s, sizeof(int64_t) * 3);
    }
    if (extra) { extra[0] = (int32_t)r_lb; extra[1] = ncand; extra[2] = n_ok_trials; }
    free(sigma); free(x_len); free(cand); free(keys); free(tmp); free(tmp2);
    topo_free(&tp);
    return OR_OK;
}

/* The seeding operators one at a time, so that each can be checked on its
 * own (Sec. 4.1.1).  or_seed_trial runs one randomized trial with R rows:
 * pi_out receives the WindowShuffle order, cellk_out the cell k in [0, R*D)
 * each sample's RandomizedBestFit gave it, layout_out the cell id r*D + d
 * after EDPAwarePair; returns 1, or 0 when best-fit found no feasible cell
 * (then cellk_out and layout_out are untouched).  or_edp_pair runs
 * EDPAwarePair alone on given completed cells. */
int or_seed_trial(const or_problem *pb, const int32_t *t, const int32_t *q, int32_t R, int32_t w,
                  uint64_t seed, uint64_t trial, int32_t *pi_out, int32_t *cellk_out,
                  int32_t *layout_out)
{
    if (check_problem(pb) || R < 1 || w < 1) return OR_INVALID;
    int32_t N = pb->n_samples;
    if ((int64_t)R * pb->n_dp > N) return OR_INVALID;
    int32_t *sigma = malloc(sizeof(int32_t) * N);
    for (int32_t i = 0; i < N; ++i) sigma[i] = i;
    g_len = t;
    qsort(sigma, N, sizeof(int32_t), cmp_len_desc);
    topo_t tp;
    topo_build(pb, &tp);
    int ok = seed_trial(pb, &tp, t, q, R, sigma, w, seed, trial, layout_out, pi_out, cellk_out);
    topo_free(&tp);
    free(sigma);
    return ok;
}

int or_edp_pair(const or_problem *pb, const int32_t *q, int32_t R, const int32_t *cellk, int32_t w,
                uint64_t seed, uint64_t trial, int32_t *layout_out)
{
    if (check_problem(pb) || R < 1 || w < 1) return OR_INVALID;
    int64_t K = (int64_t)R * pb->n_dp;
    for (int32_t i = 0; i < pb->n_samples; ++i) if (cellk[i] < 0 || cellk[i] >= K) return OR_INVALID;
    topo_t tp;
    topo_build(pb, &tp);
    edp_aware_pair(pb, &tp, q, R, cellk, w, seed, trial, layout_out);
    topo_free(&tp);
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Population annealing (Alg. 3). */

typedef struct {
    int32_t n_sweeps, steps_per_sweep;
    const double *temperatures;   /* [n_sweeps] */
    double t_next;                /* temperature of the level after this call; <= 0: final */
    uint32_t p_guide_u32, rho_u32;
    uint64_t seed;
    int32_t sweep_offset;
    int32_t init_incumbent;
} or_anneal_params;

/* Energy (Eq. pa-energy) of a fixed-point score: S_i = s_i / (2^F C). */
static double energy_of(const int64_t *s, double scale)
{
    double S0 = (double)s[0] / scale, S1 = (double)s[1] / scale, S2 = (double)s[2] / scale;
    double e = S0 + 1e-6 * S1;
    return e + 1e-9 * S2;
}

/* Exported for the tests: the energy of n score triples. */
void or_energy(int32_t n, const int64_t *s, int32_t frac_bits, int64_t capacity, double *out)
{
    double scale = (double)((int64_t)1 << frac_bits) * (double)capacity;
    for (int32_t j = 0; j < n; ++j) out[j] = energy_of(s + (int64_t)j * 3, scale);
}

/* One replica's chain state. */
typedef struct {
    int32_t *cell_of;      /* [N] */
    int32_t **mem;         /* [B] sorted member ids */
    int32_t *msize, *mcap; /* [B] */
    int64_t *T, *Q2;       /* [B] */
    int64_t *W;            /* [R*G][L][P] */
    int64_t *J;            /* [R*G] */
    int64_t *U;            /* [G] */
    int64_t s[3];
} chain_t;

typedef struct {
    const or_problem *pb;
    const topo_t *tp;
    const int32_t *t, *q;
    int32_t R;
    double scale;
} ctx_t;

static void mem_insert(chain_t *ch, int32_t c, int32_t id)
{
    if (ch->msize[c] == ch->mcap[c]) {
        ch->mcap[c] = ch->mcap[c] * 2 + 4;
        ch->mem[c] = realloc(ch->mem[c], sizeof(int32_t) * ch->mcap[c]);
    }
    int32_t k = ch->msize[c];
    while (k > 0 && ch->mem[c][k - 1] > id) { ch->mem[c][k] = ch->mem[c][k - 1]; --k; }
    ch->mem[c][k] = id;
    ch->msize[c]++;
}
static void mem_erase(chain_t *ch, int32_t c, int32_t id)
{
    int32_t k = 0;
    while (ch->mem[c][k] != id) ++k;
    for (; k + 1 < ch->msize[c]; ++k) ch->mem[c][k] = ch->mem[c][k + 1];
    ch->msize[c]--;
}

static int64_t cell_cost_sum(const ctx_t *cx, const chain_t *ch, int64_t c)
{
    int64_t a = 0;
    for (int32_t s = 0; s < cx->pb->n_stages; ++s)
        a += cx->pb->alpha_fp[s] * ch->T[c] + cx->pb->beta_fp[s] * ch->Q2[c];
    return a;
}

/* A(r,g) from the cell statistics, with the two cells c1, c2 optionally
 * replaced by the (T, Q2) values given. */
static int64_t attention_of(const ctx_t *cx, const chain_t *ch, int32_t r, int32_t g,
                            int64_t c1, int64_t T1, int64_t Q1, int64_t c2, int64_t T2, int64_t Q2v)
{
    const or_problem *pb = cx->pb;
    int32_t D = pb->n_dp;
    int64_t a = 0;
    for (int32_t s = 0; s < pb->n_stages; ++s) {
        int64_t mx = 0;
        for (int32_t k = 0; k < cx->tp->count[g]; ++k) {
            int64_t c = (int64_t)r * D + cx->tp->slots[(int64_t)g * D + k];
            int64_t T = ch->T[c], Q = ch->Q2[c];
            if (c == c1) { T = T1; Q = Q1; }
            else if (c == c2) { T = T2; Q = Q2v; }
            int64_t cost = pb->alpha_fp[s] * T + pb->beta_fp[s] * Q;
            if (k == 0 || cost > mx) mx = cost;
        }
        a += mx;
    }
    return a;
}

static int64_t expert_of_table(const ctx_t *cx, const int64_t *w)
{
    int32_t L = cx->pb->n_layers, P = cx->pb->n_ranks;
    int64_t esum = 0;
    for (int32_t l = 0; l < L; ++l) {
        int64_t mx = w[(int64_t)l * P];
        for (int32_t p = 1; p < P; ++p) if (w[(int64_t)l * P + p] > mx) mx = w[(int64_t)l * P + p];
        esum += mx;
    }
    return esum << cx->pb->frac_bits;
}

static void chain_init(const ctx_t *cx, chain_t *ch, const int32_t *layout)
{
    const or_problem *pb = cx->pb;
    int32_t N = pb->n_samples, L = pb->n_layers, P = pb->n_ranks, D = pb->n_dp, G = pb->n_edp;
    int64_t B = (int64_t)cx->R * D, RG = (int64_t)cx->R * G, LP = (int64_t)L * P;
    ch->cell_of = malloc(sizeof(int32_t) * N);
    ch->mem = calloc(B, sizeof(int32_t *));
    ch->msize = calloc(B, sizeof(int32_t));
    ch->mcap = calloc(B, sizeof(int32_t));
    ch->T = calloc(B, sizeof(int64_t));
    ch->Q2 = calloc(B, sizeof(int64_t));
    ch->W = calloc((size_t)RG * LP + 1, sizeof(int64_t));
    ch->J = calloc(RG, sizeof(int64_t));
    ch->U = calloc(G, sizeof(int64_t));
    memcpy(ch->cell_of, layout, sizeof(int32_t) * N);
    for (int32_t i = 0; i < N; ++i) {
        int32_t c = layout[i];
        mem_insert(ch, c, i);
        ch->T[c] += cx->t[i];
        ch->Q2[c] += (int64_t)cx->t[i] * cx->t[i];
        int64_t h = (int64_t)(c / D) * G + pb->dp_to_edp[c % D];
        for (int64_t x = 0; x < LP; ++x) ch->W[h * LP + x] += cx->q[(int64_t)i * LP + x];
    }
    for (int64_t h = 0; h < RG; ++h) {
        int32_t r = (int32_t)(h / G), g = (int32_t)(h % G);
        ch->J[h] = attention_of(cx, ch, r, g, -1, 0, 0, -1, 0, 0) + expert_of_table(cx, ch->W + h * LP);
        ch->U[g] += ch->J[h];
    }
    ch->s[0] = ch->s[1] = ch->s[2] = 0;
    for (int32_t g = 0; g < G; ++g) { if (g == 0 || ch->U[g] > ch->s[0]) ch->s[0] = ch->U[g]; ch->s[1] += ch->U[g]; }
    for (int64_t h = 0; h < RG; ++h) if (h == 0 || ch->J[h] > ch->s[2]) ch->s[2] = ch->J[h];
}

static void chain_free(const ctx_t *cx, chain_t *ch)
{
    int64_t B = (int64_t)cx->R * cx->pb->n_dp;
    for (int64_t c = 0; c < B; ++c) free(ch->mem[c]);
    free(ch->cell_of); free(ch->mem); free(ch->msize); free(ch->mcap);
    free(ch->T); free(ch->Q2); free(ch->W); free(ch->J); free(ch->U);
}

/* Roulette over non-negative int64 weights in index order: pick =
 * bnd(word, total) and the first index whose inclusive prefix exceeds pick;
 * all-zero weights fall back to a uniform index. */
static int64_t roulette(const int64_t *wts, int64_t n, uint64_t word)
{
    int64_t total = 0;
    for (int64_t h = 0; h < n; ++h) total += wts[h];
    if (total == 0) return (int64_t)bnd(word, (uint64_t)n);
    uint64_t pick = bnd(word, (uint64_t)total);
    int64_t pref = 0;
    for (int64_t h = 0; h < n; ++h) {
        pref += wts[h];
        if ((uint64_t)pref > pick) return h;
    }
    return n - 1; /* unreachable */
}

typedef struct {
    int64_t term[3], best[3];
    int64_t accepted, evaluated;
    int32_t *best_layout; /* [N] */
    uint8_t *step_log;    /* [K] or NULL */
    int32_t mismatch;     /* incremental != full rescore was seen */
} chain_result;

/* K fixed-temperature steps of one replica (Alg. 3, inner loop). */
static void run_chain(const ctx_t *cx, chain_t *ch, const or_anneal_params *ap, int32_t level,
                      int32_t replica, double temp, chain_result *res, int check_full)
{
    const or_problem *pb = cx->pb;
    const topo_t *tp = cx->tp;
    int32_t N = pb->n_samples, L = pb->n_layers, P = pb->n_ranks, D = pb->n_dp, G = pb->n_edp;
    int32_t R = cx->R;
    int64_t B = (int64_t)R * D, RG = (int64_t)R * G, LP = (int64_t)L * P, C = pb->capacity;
    const int32_t *t = cx->t, *q = cx->q;
    int64_t *wts = malloc(sizeof(int64_t) * (RG > D ? RG : D));
    int64_t *W1 = malloc(sizeof(int64_t) * (LP + 1)), *W2 = malloc(sizeof(int64_t) * (LP + 1));
    memcpy(res->best, ch->s, sizeof(ch->s));
    memcpy(res->best_layout, ch->cell_of, sizeof(int32_t) * N);
    res->accepted = res->evaluated = 0;
    double e_cur = energy_of(ch->s, cx->scale);
    uint64_t key[2] = {ap->seed, 0};
    for (int32_t k = 0; k < ap->steps_per_sweep; ++k) {
        uint64_t w[8];
        uint64_t c0[4] = {(uint64_t)k, (uint64_t)(uint32_t)level, (uint64_t)(uint32_t)replica, 0};
        uint64_t c1[4] = {(uint64_t)k, (uint64_t)(uint32_t)level, (uint64_t)(uint32_t)replica, 1};
        or_philox4x64(c0, key, w);
        or_philox4x64(c1, key, w + 4);
        int guided = (uint32_t)w[0] < ap->p_guide_u32;
        int reloc = (uint32_t)(w[0] >> 32) < ap->rho_u32;
        int32_t i, j = -1;
        int64_t ca, cb; /* source and target cells */
        if (guided) {
            /* GuidedProposal: source row-shard by J, source cell by its
             * attention cost, target row-shard by (J_max - J + 1). */
            int64_t h1 = roulette(ch->J, RG, w[1]);
            int32_t r1 = (int32_t)(h1 / G), g1 = (int32_t)(h1 % G);
            int32_t m1 = tp->count[g1];
            for (int32_t x = 0; x < m1; ++x)
                wts[x] = cell_cost_sum(cx, ch, (int64_t)r1 * D + tp->slots[(int64_t)g1 * D + x]);
            int64_t xi = roulette(wts, m1, w[2]);
            ca = (int64_t)r1 * D + tp->slots[(int64_t)g1 * D + xi];
            i = ch->mem[ca][bnd(w[3], (uint64_t)ch->msize[ca])];
            int64_t jmax = ch->s[2];
            for (int64_t h = 0; h < RG; ++h) wts[h] = jmax - ch->J[h] + 1;
            int64_t h2 = roulette(wts, RG, w[4]);
            int32_t r2 = (int32_t)(h2 / G), g2 = (int32_t)(h2 % G);
            cb = (int64_t)r2 * D + tp->slots[(int64_t)g2 * D + bnd(w[5], (uint64_t)tp->count[g2])];
            if (!reloc) j = ch->mem[cb][bnd(w[6], (uint64_t)ch->msize[cb])];
        } else {
            i = (int32_t)bnd(w[1], (uint64_t)N);
            ca = ch->cell_of[i];
            if (!reloc) { j = (int32_t)bnd(w[4], (uint64_t)N); cb = ch->cell_of[j]; }
            else cb = (int64_t)bnd(w[4], (uint64_t)B);
        }
        /* Feasibility (Eqs. nonempty-cell, token-capacity): an infeasible
         * proposal consumes the step without an accept test. */
        int feasible = (ca != cb);
        int64_t Ta = ch->T[ca], Tb = ch->T[cb], Qa = ch->Q2[ca], Qb = ch->Q2[cb];
        int64_t ti = t[i], tj = (j >= 0) ? t[j] : 0;
        if (feasible) {
            if (!reloc) feasible = (Ta - ti + tj <= C) && (Tb - tj + ti <= C);
            else feasible = (ch->msize[ca] >= 2) && (Tb + ti <= C);
        }
        if (!feasible) { if (res->step_log) res->step_log[k] = 0; continue; }
        res->evaluated++;
        /* IncrementalScore: new statistics of the two cells and new tables
         * of the two row-shards, then the exact score. */
        int64_t nTa = Ta - ti + tj, nTb = Tb + ti - tj;
        int64_t nQa = Qa - ti * ti + tj * tj, nQb = Qb + ti * ti - tj * tj;
        int32_t ra = (int32_t)(ca / D), ga = pb->dp_to_edp[ca % D];
        int32_t rb = (int32_t)(cb / D), gb = pb->dp_to_edp[cb % D];
        int64_t ha = (int64_t)ra * G + ga, hb = (int64_t)rb * G + gb;
        int64_t Ja, Jb;
        if (ha == hb) {
            int64_t ea = ch->J[ha] - attention_of(cx, ch, ra, ga, -1, 0, 0, -1, 0, 0);
            Ja = attention_of(cx, ch, ra, ga, ca, nTa, nQa, cb, nTb, nQb) + ea;
            Jb = Ja;
        } else {
            for (int64_t x = 0; x < LP; ++x) {
                int64_t qi = q[(int64_t)i * LP + x], qj = (j >= 0) ? q[(int64_t)j * LP + x] : 0;
                W1[x] = ch->W[ha * LP + x] - qi + qj;
                W2[x] = ch->W[hb * LP + x] + qi - qj;
            }
            Ja = attention_of(cx, ch, ra, ga, ca, nTa, nQa, -1, 0, 0) + expert_of_table(cx, W1);
            Jb = attention_of(cx, ch, rb, gb, cb, nTb, nQb, -1, 0, 0) + expert_of_table(cx, W2);
        }
        int64_t ns[3] = {0, 0, 0};
        for (int32_t g = 0; g < G; ++g) {
            int64_t U = ch->U[g];
            if (g == ga) U += Ja - ch->J[ha];
            if (g == gb && hb != ha) U += Jb - ch->J[hb];
            if (g == 0 || U > ns[0]) ns[0] = U;
            ns[1] += U;
        }
        for (int64_t h = 0; h < RG; ++h) {
            int64_t Jh = (h == ha) ? Ja : (h == hb) ? Jb : ch->J[h];
            if (h == 0 || Jh > ns[2]) ns[2] = Jh;
        }
        /* Metropolis test (Alg. 3): a lexicographic improvement, or
         * u < exp(-max(Delta, 0) / T_n). */
        double e_new = energy_of(ns, cx->scale);
        double denom = fabs(e_cur) > 1.0 ? fabs(e_cur) : 1.0;
        double delta = (e_new - e_cur) / denom;
        double z = (delta > 0.0 ? delta : 0.0) / temp;
        double u = (double)(uint32_t)(w[7] >> 32) * (1.0 / 4294967296.0);
        int accept = lex_lt(ns, ch->s) || (u < or_exp_det(-z));
        if (!accept) { if (res->step_log) res->step_log[k] = 1; continue; }
        if (res->step_log) res->step_log[k] = 2;
        res->accepted++;
        /* Commit. */
        ch->cell_of[i] = (int32_t)cb;
        mem_erase(ch, (int32_t)ca, i);
        mem_insert(ch, (int32_t)cb, i);
        if (j >= 0) {
            ch->cell_of[j] = (int32_t)ca;
            mem_erase(ch, (int32_t)cb, j);
            mem_insert(ch, (int32_t)ca, j);
        }
        ch->T[ca] = nTa; ch->Q2[ca] = nQa; ch->T[cb] = nTb; ch->Q2[cb] = nQb;
        if (ha != hb) {
            memcpy(ch->W + ha * LP, W1, sizeof(int64_t) * LP);
            memcpy(ch->W + hb * LP, W2, sizeof(int64_t) * LP);
        }
        ch->U[ga] += Ja - ch->J[ha];
        ch->J[ha] = Ja;
        if (hb != ha) { ch->U[gb] += Jb - ch->J[hb]; ch->J[hb] = Jb; }
        memcpy(ch->s, ns, sizeof(ns));
        e_cur = e_new;
        if (check_full) {
            int64_t fs[3];
            or_score(pb, t, q, R, ch->cell_of, fs, NULL, NULL, NULL);
            if (fs[0] != ch->s[0] || fs[1] != ch->s[1] || fs[2] != ch->s[2]) res->mismatch = 1;
        }
        if (lex_lt(ch->s, res->best)) {
            memcpy(res->best, ch->s, sizeof(ch->s));
            memcpy(res->best_layout, ch->cell_of, sizeof(int32_t) * N);
        }
    }
    memcpy(res->term, ch->s, sizeof(ch->s));
    free(wts); free(W1); free(W2);
}

typedef struct {
    const ctx_t *cx;
    const or_anneal_params *ap;
    int32_t level, pop, tid, nthreads;
    double temp;
    int32_t *layouts;        /* [pop][N] in: start states, out: terminal states */
    chain_result *res;
    int check_full;
    const int32_t *replica_ids;  /* member j runs the chain of replica replica_ids[j] */
} worker_arg;

static void *worker(void *p)
{
    worker_arg *a = p;
    int32_t N = a->cx->pb->n_samples;
    for (int32_t j = a->tid; j < a->pop; j += a->nthreads) {
        chain_t ch;
        chain_init(a->cx, &ch, a->layouts + (size_t)j * N);
        int32_t rid = a->replica_ids ? a->replica_ids[j] : j;
        run_chain(a->cx, &ch, a->ap, a->level, rid, a->temp, &a->res[j], a->check_full);
        memcpy(a->layouts + (size_t)j * N, ch.cell_of, sizeof(int32_t) * N);
        chain_free(a->cx, &ch);
    }
    return NULL;
}

/* Systematic resampling (Alg. 3, the level boundary), in exact arithmetic on
 * quantised weights: w_j = floor(2^40 exp(-(1/T_next - 1/T_cur) E~_j)) with
 * E~_j = (E_j - E_min) / max(|E_min|, 1); F = inclusive prefix; with u0 drawn
 * as V / (2^32 P), member m takes parent min{ j : F_j / F_{P-1} >= u0 + m/P }. */
void or_resample_at(int32_t pop, const double *energies, double t_cur, double t_next,
                    uint64_t V, int32_t *parent);

void or_resample(int32_t pop, const double *energies, double t_cur, double t_next,
                 uint64_t seed, int32_t level, int32_t *parent)
{
    uint64_t ctr[4] = {0, (uint64_t)(uint32_t)level, 0xFFFFFFFFull, 2}, key[2] = {seed, 0}, out[4];
    or_philox4x64(ctr, key, out);
    or_resample_at(pop, energies, t_cur, t_next, out[0] >> 32, parent);
}

/* The same step for a given V in [0, 2^32) (u0 = V / (2^32 P)). */
void or_resample_at(int32_t pop, const double *energies, double t_cur, double t_next,
                    uint64_t V, int32_t *parent)
{
    double emin = energies[0];
    for (int32_t j = 1; j < pop; ++j) if (energies[j] < emin) emin = energies[j];
    double denom = fabs(emin) > 1.0 ? fabs(emin) : 1.0;
    double cfac = (1.0 / t_next) - (1.0 / t_cur);
    uint64_t *F = malloc(sizeof(uint64_t) * pop);
    uint64_t acc = 0;
    for (int32_t j = 0; j < pop; ++j) {
        double en = (energies[j] - emin) / denom;
        double wh = or_exp_det(-(cfac * en));
        uint64_t wq = (uint64_t)floor(ldexp(wh, 40));
        acc += wq;
        F[j] = acc;
    }
    uint64_t S = F[pop - 1];
    for (int32_t m = 0; m < pop; ++m) {
        unsigned __int128 rhs = (unsigned __int128)S * (V + ((uint64_t)m << 32));
        int32_t j = 0;
        while (!((unsigned __int128)F[j] * (uint64_t)pop * ((uint64_t)1 << 32) >= rhs)) ++j;
        parent[m] = j;
    }
    free(F);
}

/* Population annealing over n_sweeps levels (Alg. 3).
 * population[pop][N]: in the start population of level sweep_offset; out the
 *   population that level sweep_offset + n_sweeps starts from (resampled when
 *   t_next > 0, terminal states otherwise).
 * best_layout[N], best_score[3]: the incumbent x*, initialised here from the
 *   population (lowest-index argmin) when init_incumbent != 0.
 * trace[n_sweeps][pop][8] (optional): terminal score, trajectory-best score,
 *   accepted count, evaluated count.  parents[n_sweeps][pop] (optional):
 *   parent of each member after the level (or -1 when no resampling).
 * step_log[n_sweeps][pop][K] (optional): 0 infeasible, 1 rejected, 2 accepted.
 * check_full: assert incremental == full rescore after every accepted step.
 * replica_ids (optional): member j draws the random stream of replica
 *   replica_ids[j] -- lets a subset of a large population be recomputed. */
int or_anneal(const or_problem *pb, const int32_t *t, const int32_t *q, int32_t R, int32_t pop,
              int32_t *population, const or_anneal_params *ap, int32_t *best_layout,
              int64_t *best_score, int64_t *trace, int32_t *parents, uint8_t *step_log,
              int32_t n_threads, int32_t check_full, const int32_t *replica_ids)
{
    int rc = check_problem(pb);
    if (rc) return rc;
    if (pop < 1 || R < 1 || ap->n_sweeps < 0 || ap->steps_per_sweep < 0) return OR_INVALID;
    for (int32_t n = 0; n < ap->n_sweeps; ++n) {
        if (!(ap->temperatures[n] > 0.0)) return OR_INVALID;
        if (n > 0 && !(ap->temperatures[n] < ap->temperatures[n - 1])) return OR_INVALID;
    }
    if (ap->n_sweeps > 0 && ap->t_next > 0.0 && !(ap->t_next < ap->temperatures[ap->n_sweeps - 1]))
        return OR_INVALID;
    if ((rc = overflow_check(pb, t, q, R, NULL))) return rc;
    int32_t N = pb->n_samples;
    topo_t tp;
    topo_build(pb, &tp);
    ctx_t cx = {pb, &tp, t, q, R, (double)((int64_t)1 << pb->frac_bits) * (double)pb->capacity};
    /* Validate the population. */
    int64_t (*sc)[3] = malloc(sizeof(int64_t[3]) * pop);
    for (int32_t j = 0; j < pop; ++j)
        if (or_score(pb, t, q, R, population + (size_t)j * N, sc[j], NULL, NULL, NULL) != 0) {
            free(sc); topo_free(&tp); return OR_LAYOUT;
        }
    if (ap->init_incumbent) {
        int32_t b = 0;
        for (int32_t j = 1; j < pop; ++j) if (lex_lt(sc[j], sc[b])) b = j;
        memcpy(best_layout, population + (size_t)b * N, sizeof(int32_t) * N);
        memcpy(best_score, sc[b], sizeof(int64_t) * 3);
    } else {
        int64_t s[3];
        if (or_score(pb, t, q, R, best_layout, s, NULL, NULL, NULL) != 0) { free(sc); topo_free(&tp); return OR_LAYOUT; }
        if (s[0] != best_score[0] || s[1] != best_score[1] || s[2] != best_score[2]) { free(sc); topo_free(&tp); return OR_LAYOUT; }
    }
    int64_t seed_best[3];
    memcpy(seed_best, sc[0], sizeof(seed_best));
    for (int32_t j = 1; j < pop; ++j) if (lex_lt(sc[j], seed_best)) memcpy(seed_best, sc[j], sizeof(seed_best));
    if (lex_lt(best_score, seed_best)) memcpy(seed_best, best_score, sizeof(seed_best));
    free(sc);
    if (n_threads < 1) n_threads = 1;
    chain_result *res = calloc(pop, sizeof(chain_result));
    for (int32_t j = 0; j < pop; ++j) res[j].best_layout = malloc(sizeof(int32_t) * N);
    int32_t *terminal = malloc(sizeof(int32_t) * (size_t)pop * N);
    int32_t *parent = malloc(sizeof(int32_t) * pop);
    double *en = malloc(sizeof(double) * pop);
    pthread_t *th = malloc(sizeof(pthread_t) * n_threads);
    worker_arg *wa = malloc(sizeof(worker_arg) * n_threads);
    int32_t K = ap->steps_per_sweep;
    for (int32_t n = 0; n < ap->n_sweeps; ++n) {
        int32_t level = ap->sweep_offset + n;
        memcpy(terminal, population, sizeof(int32_t) * (size_t)pop * N);
        for (int32_t j = 0; j < pop; ++j)
            res[j].step_log = step_log ? step_log + ((size_t)n * pop + j) * K : NULL;
        for (int32_t x = 0; x < n_threads; ++x) {
            wa[x] = (worker_arg){&cx, ap, level, pop, x, n_threads, ap->temperatures[n], terminal, res,
                                 check_full, replica_ids};
            pthread_create(&th[x], NULL, worker, &wa[x]);
        }
        for (int32_t x = 0; x < n_threads; ++x) pthread_join(th[x], NULL);
        /* Incumbent: strict improvements, members in ascending order. */
        for (int32_t j = 0; j < pop; ++j)
            if (lex_lt(res[j].best, best_score)) {
                memcpy(best_score, res[j].best, sizeof(int64_t) * 3);
                memcpy(best_layout, res[j].best_layout, sizeof(int32_t) * N);
            }
        if (trace)
            for (int32_t j = 0; j < pop; ++j) {
                int64_t *tr = trace + ((size_t)n * pop + j) * 8;
                tr[0] = res[j].term[0]; tr[1] = res[j].term[1]; tr[2] = res[j].term[2];
                tr[3] = res[j].best[0]; tr[4] = res[j].best[1]; tr[5] = res[j].best[2];
                tr[6] = res[j].accepted; tr[7] = res[j].evaluated;
            }
        double t_after = (n + 1 < ap->n_sweeps) ? ap->temperatures[n + 1] : ap->t_next;
        if (t_after > 0.0) {
            for (int32_t j = 0; j < pop; ++j) en[j] = energy_of(res[j].term, cx.scale);
            or_resample(pop, en, ap->temperatures[n], t_after, ap->seed, level, parent);
            for (int32_t m = 0; m < pop; ++m)
                memcpy(population + (size_t)m * N, terminal + (size_t)parent[m] * N, sizeof(int32_t) * N);
        } else {
            for (int32_t m = 0; m < pop; ++m) parent[m] = -1;
            memcpy(population, terminal, sizeof(int32_t) * (size_t)pop * N);
        }
        if (parents) memcpy(parents + (size_t)n * pop, parent, sizeof(int32_t) * pop);
    }
    /* Validate x* and check non-regression against the start population. */
    int64_t fs[3];
    int st = or_score(pb, t, q, R, best_layout, fs, NULL, NULL, NULL);
    rc = OR_OK;
    if (st != 0 || fs[0] != best_score[0] || fs[1] != best_score[1] || fs[2] != best_score[2]) rc = OR_INTERNAL;
    if (lex_lt(seed_best, best_score)) rc = OR_INTERNAL;
    for (int32_t j = 0; j < pop; ++j) if (res[j].mismatch) rc = OR_INTERNAL;
    for (int32_t j = 0; j < pop; ++j) free(res[j].best_layout);
    free(res); free(terminal); free(parent); free(en); free(th); free(wa);
    topo_free(&tp);
    return rc;
}
