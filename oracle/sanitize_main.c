/*
 * Sanitizer driver for the CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * Built by tests/test_oracle_sanitize.py with gcc under AddressSanitizer and
 * UndefinedBehaviorSanitizer (and, separately, ThreadSanitizer for the
 * threaded annealing workers).  It includes the oracle's single source file
 * and runs every exported function on small windows with one and two EDP
 * shards and one and two attention stages; a sanitizer report aborts the run,
 * and a return code other than the expected one exits non-zero.
 *
 * The window is drawn with a local xorshift64* generator: lengths uniform in
 * [16, 400], each sample's k * t routed tokens spread over the experts with no
 * expert above t.  Nothing here checks values (the pins do); it only drives
 * the code paths.
 */
#include "routepack_oracle.c"

#include <stdio.h>

static uint64_t rng_state = 0x9E3779B97F4A7C15ULL;
static uint64_t rnd(void)
{
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return rng_state * 0x2545F4914F6CDD1DULL;
}
static int32_t rnd_in(int32_t lo, int32_t hi) { return lo + (int32_t)(rnd() % (uint64_t)(hi - lo + 1)); }

#define CHECK(cond, what)                                                   \
    do {                                                                    \
        if (!(cond)) { fprintf(stderr, "sanitize_main: %s failed\n", what); \
                       return 1; }                                          \
    } while (0)

static int run_case(int32_t G, int32_t S, int32_t n_threads)
{
    const int32_t N = 48, L = 3, E = 8, P = 4, K = 2, D = 4;
    int32_t dp_to_edp[4];
    for (int32_t d = 0; d < D; ++d) dp_to_edp[d] = (G == 1) ? 0 : d / (D / G);
    int64_t alpha[2] = {4096, 2048}, beta[2] = {0, 1};
    if (S == 1) { alpha[0] = 4096; beta[0] = 1; }
    or_problem pb = {N, L, E, K, P, D, G, dp_to_edp, 1024, S, alpha, beta, 12, 1};

    int32_t *t = malloc(sizeof(int32_t) * N);
    int32_t *demand = calloc((size_t)N * L * E, sizeof(int32_t));
    for (int32_t i = 0; i < N; ++i) {
        t[i] = rnd_in(16, 400);
        for (int32_t l = 0; l < L; ++l) {
            int32_t *a = demand + ((int64_t)i * L + l) * E;
            for (int64_t tok = 0; tok < (int64_t)K * t[i]; ++tok) {
                int32_t e;
                do { e = rnd_in(0, E - 1); } while (a[e] >= t[i]);
                a[e]++;
            }
        }
    }
    int64_t *agg = malloc(sizeof(int64_t) * L * E);
    int32_t *slot = malloc(sizeof(int32_t) * L * E);
    int64_t *load = malloc(sizeof(int64_t) * L * P);
    int32_t *q = malloc(sizeof(int32_t) * N * L * P);
    or_aggregate(N, L, E, demand, agg);
    CHECK(or_place(L, E, P, agg, slot, load) == OR_OK, "or_place");
    CHECK(or_project(N, L, E, P, demand, slot, q) == OR_OK, "or_project");

    const int32_t pop = 8;
    int32_t r_star = 0, cert = 0, extra[3];
    int32_t *popl = malloc(sizeof(int32_t) * pop * N);
    int64_t *sc = malloc(sizeof(int64_t) * pop * 3);
    CHECK(or_pack_rows(&pb, t, q, 2000, 8, 3, pop, &r_star, &cert, popl, sc, extra) == OR_OK, "or_pack_rows");

    int64_t s[3], J[64];
    double diag[8];
    CHECK(or_score(&pb, t, q, r_star, popl, s, J, diag, load) == 0, "or_score");
    int32_t bad = popl[0];
    popl[0] = r_star * D;      /* out of range: a status bit, no error */
    CHECK(or_score(&pb, t, q, r_star, popl, s, NULL, NULL, NULL) != 0, "or_score status");
    popl[0] = bad;

    int32_t *pi = malloc(sizeof(int32_t) * N), *ck = malloc(sizeof(int32_t) * N);
    int32_t *lay = malloc(sizeof(int32_t) * N);
    CHECK(or_seed_trial(&pb, t, q, r_star, 3, 2000, 1, pi, ck, lay) >= 0, "or_seed_trial");
    for (int32_t i = 0; i < N; ++i) ck[i] = i % (r_star * D);
    CHECK(or_edp_pair(&pb, q, r_star, ck, 2, 2000, 1, lay) == OR_OK, "or_edp_pair");

    const int32_t levels = 4, steps = 64;
    double temps[4] = {1e-3, 5e-4, 2e-4, 1e-4};
    or_anneal_params ap = {levels, steps, temps, 5e-5, 0xCCCCCCCDu, 0x40000000u, 1000, 0, 1};
    int32_t *best = malloc(sizeof(int32_t) * N);
    int64_t bs[3];
    int64_t *trace = malloc(sizeof(int64_t) * levels * pop * 8);
    int32_t *par = malloc(sizeof(int32_t) * levels * pop);
    uint8_t *slog = malloc((size_t)levels * pop * steps);
    CHECK(or_anneal(&pb, t, q, r_star, pop, popl, &ap, best, bs, trace, par, slog, n_threads, 1, NULL) == OR_OK,
          "or_anneal");
    or_anneal_params ap2 = {2, steps, temps, 0.0, 0xCCCCCCCDu, 0x40000000u, 1000, levels, 0};
    int32_t rid[8] = {7, 6, 5, 4, 3, 2, 1, 0};
    CHECK(or_anneal(&pb, t, q, r_star, pop, popl, &ap2, best, bs, NULL, NULL, NULL, n_threads, 0, rid) == OR_OK,
          "or_anneal resume");

    double en[8];
    int32_t parent[8];
    for (int32_t j = 0; j < pop; ++j) en[j] = 1.0 + 1e-4 * (double)j;
    or_resample(pop, en, 1e-3, 5e-4, 1000, 3, parent);
    or_resample_at(pop, en, 1e-3, 5e-4, 0, parent);

    free(t); free(demand); free(agg); free(slot); free(load); free(q); free(popl); free(sc);
    free(pi); free(ck); free(lay); free(best); free(trace); free(par); free(slog);
    return 0;
}

int main(void)
{
    uint64_t ctr[4] = {1, 2, 3, 4}, key[2] = {5, 6}, out[4];
    or_philox4x64(ctr, key, out);
    volatile double e = or_exp_det(-3.5) + or_exp_det(-800.0) + or_exp_det(0.0);
    (void)e;
    for (int32_t G = 1; G <= 2; ++G)
        for (int32_t S = 1; S <= 2; ++S)
            if (run_case(G, S, G == 1 ? 1 : 4)) return 1;
    printf("sanitize_main ok\n");
    return 0;
}
