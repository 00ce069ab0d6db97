// Fixed-row population annealing (Alg. 3) on gfx950.
//
// One workgroup (4 waves) runs one population member for the K steps of a
// temperature level.  Replica state lives in a per-member slab in HBM
// (double-buffered across levels, so resampling is a gather at the start of
// the next level):
//   cell_of [N]         cell id of every sample
//   pool    [N]         sample ids sorted by (cell, id); cell c's members are
//                       pool[start[c] .. start[c+1])
//   start   [B+1]
//   T, Q2   [B] int64   sum t and sum t^2 of every cell
//   W       [R*G][L][P] int32 row-shard expert loads (Eq. row-expert-load)
//   J, A    [R*G] int64 joint cost and attention part per row-shard
// During the level, W is staged in LDS when it fits.  Every W entry is
// private to one thread: thread tid owns entries e = tid + 256 m of every
// row, so the incremental update of two rows (2*L*P entries) and its commit
// need no barrier; the per-layer max over P ranks is a segmented wave
// reduction over P adjacent lanes.  J, A and U are replicated in the
// registers of each wave, so proposal selection (roulettes over J and cell
// attention) runs on every wave without communication.  The only block
// barriers are the cross-wave sum of the two E' partials of a feasible
// proposal and the commit of an accepted one.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "rp_anneal.h"
#include "rp_device.h"
#include "rp_internal.h"

namespace rp {

int eval_layouts(const routepack_problem *p, const Topology &topo, const DeviceProblem &dp,
                 const int32_t *t, const int32_t *q, int32_t R, int64_t n, const int32_t *layouts,
                 int64_t *scores, int32_t *status, int64_t *J, double *diag,
                 const int64_t *rank_load, hipStream_t stream);
__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t v);

template <bool WLDS>
__global__ void __launch_bounds__(kThreads) k_anneal_level(AnnealArgs a) {
    extern __shared__ char smem[];
    const int tid = threadIdx.x, lane = lane_id(), wv = wave_id();
    const int m = blockIdx.x;
    const int par = a.parent ? a.parent[m] : m;
    char *src = a.src + (int64_t)par * a.off.bytes;
    char *dst = a.dst + (int64_t)m * a.off.bytes;
    int64_t *red = reinterpret_cast<int64_t *>(smem);  // [2][4][2]
    int32_t *Wl = reinterpret_cast<int32_t *>(smem + 128);

    const int32_t N = a.N, B = a.B, RG = a.RG, LP = a.LP, D = a.D, G = a.G;
    int32_t *cell_of = at<int32_t>(dst, a.off.cell);
    int32_t *pool = at<int32_t>(dst, a.off.pool);
    int32_t *start = at<int32_t>(dst, a.off.start);
    int64_t *T = at<int64_t>(dst, a.off.T);
    int64_t *Q = at<int64_t>(dst, a.off.Q);
    int32_t *Wg = at<int32_t>(dst, a.off.W);

    // Prologue: gather the parent's terminal state.
    {
        const int32_t *s_cell = at<int32_t>(src, a.off.cell), *s_pool = at<int32_t>(src, a.off.pool);
        for (int32_t x = tid; x < N; x += kThreads) {
            cell_of[x] = s_cell[x];
            pool[x] = s_pool[x];
        }
        const int32_t *s_start = at<int32_t>(src, a.off.start);
        for (int32_t x = tid; x <= B; x += kThreads) start[x] = s_start[x];
        const int64_t *s_T = at<int64_t>(src, a.off.T), *s_Q = at<int64_t>(src, a.off.Q);
        for (int32_t x = tid; x < B; x += kThreads) {
            T[x] = s_T[x];
            Q[x] = s_Q[x];
        }
        const int32_t *s_W = at<int32_t>(src, a.off.W);
        for (int64_t h = 0; h < RG; ++h)
            for (int x = 0; x < a.nx; ++x) {
                const int32_t e = tid + kThreads * x;
                if (e < LP) {
                    if (WLDS) Wl[h * LP + e] = s_W[h * LP + e];
                    else Wg[h * LP + e] = s_W[h * LP + e];
                }
            }
    }
    // Per-wave registers: J, A for h = lane + 64 x; U for g = lane.
    int64_t Jr[kMaxJPL], Ar[kMaxJPL];
    {
        const int64_t *s_J = at<int64_t>(src, a.off.J), *s_A = at<int64_t>(src, a.off.A);
#pragma unroll
        for (int x = 0; x < kMaxJPL; ++x) {
            const int h = x * kWave + lane;
            Jr[x] = h < RG ? s_J[h] : 0;
            Ar[x] = h < RG ? s_A[h] : 0;
        }
        if (tid < RG) {
            at<int64_t>(dst, a.off.J)[tid] = s_J[tid];
            at<int64_t>(dst, a.off.A)[tid] = s_A[tid];
        }
        for (int h = tid + kThreads; h < RG; h += kThreads) {
            at<int64_t>(dst, a.off.J)[h] = s_J[h];
            at<int64_t>(dst, a.off.A)[h] = s_A[h];
        }
    }
    int64_t Ur = 0;
    if (lane < G)
        for (int r = 0; r < a.R; ++r) Ur += at<int64_t>(src, a.off.J)[(int64_t)r * G + lane];
    int64_t s0 = wave_max(lane < G ? Ur : LLONG_MIN);
    int64_t s1 = wave_sum(lane < G ? Ur : 0);
    int64_t s2 = LLONG_MIN;
#pragma unroll
    for (int x = 0; x < kMaxJPL; ++x) {
        const int h = x * kWave + lane;
        if (h < RG) s2 = Jr[x] > s2 ? Jr[x] : s2;
    }
    s2 = wave_max(s2);
    __syncthreads();

    int64_t b0 = s0, b1 = s1, b2 = s2;
    int32_t best_is_start = 1;
    int64_t n_acc = 0, n_eval = 0;
    double e_cur = energy(s0, s1, s2, a.scale);
    uint64_t rw0 = 0, rw1 = 0, rw2 = 0, rw3 = 0;
    const int32_t P = a.P;

    for (int k = 0; k < a.K; ++k) {
        if ((k & 31) == 0) {
            // 32 steps x 2 blocks of Philox words, one block per lane.
            const U64x4 blk = philox4x64_10((uint64_t)(k + (lane >> 1)), (uint64_t)(uint32_t)a.level,
                                            (uint64_t)(uint32_t)m, (uint64_t)(lane & 1), a.seed, 0);
            rw0 = blk.v[0];
            rw1 = blk.v[1];
            rw2 = blk.v[2];
            rw3 = blk.v[3];
        }
        const int ls = 2 * (k & 31);
        const uint64_t w0 = readlane64(rw0, ls), w1 = readlane64(rw1, ls);
        const uint64_t w2 = readlane64(rw2, ls), w3 = readlane64(rw3, ls);
        const uint64_t w4 = readlane64(rw0, ls + 1), w5 = readlane64(rw1, ls + 1);
        const uint64_t w6 = readlane64(rw2, ls + 1), w7 = readlane64(rw3, ls + 1);
        const bool guided = (uint32_t)w0 < a.p_guide;
        const bool reloc = (uint32_t)(w0 >> 32) < a.rho;
        int32_t i, j = -1, c1, c2, pos_i = -1, pos_j = -1;
        if (guided) {
            const int h1 = roulette_chunks<kMaxJPL>(Jr, RG, w1, s1);
            const int32_t r1 = h1 / G, g1 = h1 % G;
            const int32_t cnt1 = a.count[g1];
            int64_t wa = 0;
            if (lane < cnt1) {
                const int32_t c = r1 * D + a.slots[g1 * D + lane];
                const int64_t tv = T[c], qv = Q[c];
                for (int s = 0; s < a.S; ++s) wa += a.alpha[s] * tv + a.beta[s] * qv;
            }
            int64_t wtmp[1] = {wa};
            const int xi = roulette_chunks<1>(wtmp, cnt1, w2, wave_sum(wa));
            c1 = r1 * D + a.slots[g1 * D + xi];
            const int32_t st1 = start[c1], sz1 = start[c1 + 1] - st1;
            pos_i = clampi(st1 + (int32_t)bounded(w3, (uint64_t)sz1), 0, N - 1);
            i = clampi(pool[pos_i], 0, N - 1);
            int64_t wt[kMaxJPL];
#pragma unroll
            for (int x = 0; x < kMaxJPL; ++x) wt[x] = s2 - Jr[x] + 1;
            const int64_t ttot = (int64_t)RG * (s2 + 1) - s1;
            const int h2 = roulette_chunks<kMaxJPL>(wt, RG, w4, ttot);
            const int32_t r2 = h2 / G, g2 = h2 % G;
            c2 = r2 * D + a.slots[g2 * D + (int32_t)bounded(w5, (uint64_t)a.count[g2])];
            if (!reloc) {
                const int32_t st2 = start[c2], sz2 = start[c2 + 1] - st2;
                pos_j = clampi(st2 + (int32_t)bounded(w6, (uint64_t)sz2), 0, N - 1);
                j = clampi(pool[pos_j], 0, N - 1);
            }
        } else {
            i = (int32_t)bounded(w1, (uint64_t)N);
            c1 = clampi(cell_of[i], 0, B - 1);
            if (!reloc) {
                j = (int32_t)bounded(w4, (uint64_t)N);
                c2 = clampi(cell_of[j], 0, B - 1);
            } else {
                c2 = (int32_t)bounded(w4, (uint64_t)B);
            }
        }
        // Feasibility: distinct cells, capacity, no emptied cell.
        bool feasible = c1 != c2;
        const int64_t T1 = T[c1], T2 = T[c2], Q1 = Q[c1], Q2v = Q[c2];
        const int64_t ti = a.t[i], tj = j >= 0 ? a.t[j] : 0;
        const int32_t sz1 = start[c1 + 1] - start[c1];
        if (feasible) {
            if (!reloc) feasible = (T1 - ti + tj <= a.C) && (T2 - tj + ti <= a.C);
            else feasible = (sz1 >= 2) && (T2 + ti <= a.C);
        }
        if (!feasible) {
            if (a.step_log && tid == 0) a.step_log[(int64_t)m * a.K + k] = 0;
            continue;
        }
        n_eval += 1;
        // IncrementalScore.
        const int64_t nT1 = T1 - ti + tj, nT2 = T2 + ti - tj;
        const int64_t nQ1 = Q1 - ti * ti + tj * tj, nQ2 = Q2v + ti * ti - tj * tj;
        const int32_t ra = c1 / D, ga = a.slot_shard[c1 % D];
        const int32_t rb = c2 / D, gb = a.slot_shard[c2 % D];
        const int32_t ha = ra * G + ga, hb = rb * G + gb;
        int64_t Aa, Ab;
        if (ha == hb) {
            Aa = attention_rs(a, T, Q, ra, ga, c1, nT1, nQ1, c2, nT2, nQ2);
            Ab = Aa;
        } else {
            Aa = attention_rs(a, T, Q, ra, ga, c1, nT1, nQ1, -1, 0, 0);
            Ab = attention_rs(a, T, Q, rb, gb, c2, nT2, nQ2, -1, 0, 0);
        }
        int32_t nwa[kMaxEPT], nwb[kMaxEPT];
        int64_t suma = 0, sumb = 0;
        if (ha != hb) {
            const int32_t *qi = a.q + (int64_t)i * LP;
            const int32_t *qj = j >= 0 ? a.q + (int64_t)j * LP : nullptr;
            const int32_t *Wa = WLDS ? Wl + (int64_t)ha * LP : Wg + (int64_t)ha * LP;
            const int32_t *Wb = WLDS ? Wl + (int64_t)hb * LP : Wg + (int64_t)hb * LP;
#pragma unroll
            for (int x = 0; x < kMaxEPT; ++x) {
                if (x < a.nx) {
                    const int32_t e = tid + kThreads * x;
                    int32_t va = INT32_MIN, vb = INT32_MIN;
                    if (e < LP) {
                        const int32_t d = qi[e] - (qj ? qj[e] : 0);
                        va = Wa[e] - d;
                        vb = Wb[e] + d;
                    }
                    nwa[x] = va;
                    nwb[x] = vb;
                    const int32_t ma = seg_max32(va, P), mb = seg_max32(vb, P);
                    if (e < LP && (lane & (P - 1)) == 0) {
                        suma += ma;
                        sumb += mb;
                    }
                }
            }
        }
        suma = wave_sum(suma);
        sumb = wave_sum(sumb);
        const int slot = (int)(n_eval & 1);
        if (lane == 0) {
            red[(slot * 4 + wv) * 2 + 0] = suma;
            red[(slot * 4 + wv) * 2 + 1] = sumb;
        }
        __syncthreads();
        int64_t Ja, Jb;
        // old J / A of the two row-shards from the wave registers
        int64_t Jha = 0, Jhb = 0, Aha = 0;
#pragma unroll
        for (int x = 0; x < kMaxJPL; ++x) {
            const int h = x * kWave + lane;
            if (h == ha) {
                Jha = Jr[x];
                Aha = Ar[x];
            }
            if (h == hb) Jhb = Jr[x];
        }
        Jha = wave_sum(Jha);
        Jhb = wave_sum(Jhb);
        Aha = wave_sum(Aha);
        if (ha == hb) {
            Ja = Aa + (Jha - Aha);
            Jb = Ja;
        } else {
            int64_t ea = 0, eb = 0;
            for (int w = 0; w < kThreads / kWave; ++w) {
                ea += red[(slot * 4 + w) * 2 + 0];
                eb += red[(slot * 4 + w) * 2 + 1];
            }
            Ja = Aa + (ea << a.F);
            Jb = Ab + (eb << a.F);
        }
        // New score.
        int64_t Un = Ur;
        if (lane == ga) Un += Ja - Jha;
        if (lane == gb && hb != ha) Un += Jb - Jhb;
        const int64_t n0 = wave_max(lane < G ? Un : LLONG_MIN);
        const int64_t n1 = s1 + (Ja - Jha) + (hb != ha ? (Jb - Jhb) : 0);
        int64_t n2 = LLONG_MIN;
#pragma unroll
        for (int x = 0; x < kMaxJPL; ++x) {
            const int h = x * kWave + lane;
            if (h < RG) {
                const int64_t v = h == ha ? Ja : (h == hb ? Jb : Jr[x]);
                n2 = v > n2 ? v : n2;
            }
        }
        n2 = wave_max(n2);
        // Metropolis test.
        const double e_new = energy(n0, n1, n2, a.scale);
        const double den = fabs(e_cur) > 1.0 ? fabs(e_cur) : 1.0;
        const double delta = (e_new - e_cur) / den;
        const double z = (delta > 0.0 ? delta : 0.0) / a.temp;
        const double u = (double)(uint32_t)(w7 >> 32) * (1.0 / 4294967296.0);
        const bool accept = lex_less(n0, n1, n2, s0, s1, s2) || (u < exp_det(-z));
        if (!accept) {
            if (a.step_log && tid == 0) a.step_log[(int64_t)m * a.K + k] = 1;
            continue;
        }
        if (a.step_log && tid == 0) a.step_log[(int64_t)m * a.K + k] = 2;
        n_acc += 1;
        // Commit: positions first (reads), then writes.
        const int32_t stc1 = start[c1], stc2 = start[c2];
        const int32_t enc1 = start[c1 + 1], enc2 = start[c2 + 1];
        if (pos_i < 0) pos_i = stc1 + seg_count_less(pool, stc1, enc1, i, -1, N);
        int32_t to1, to2 = 0;
        if (!reloc) {
            if (pos_j < 0) pos_j = stc2 + seg_count_less(pool, stc2, enc2, j, -1, N);
            to1 = stc1 + seg_count_less(pool, stc1, enc1, j, i, N);
            to2 = stc2 + seg_count_less(pool, stc2, enc2, i, j, N);
        } else {
            const int32_t rk = seg_count_less(pool, stc2, enc2, i, -1, N);
            to1 = (c1 < c2) ? (stc2 - 1 + rk) : (stc2 + rk);
        }
        pos_i = clampi(pos_i, 0, N - 1);
        pos_j = clampi(pos_j, 0, N - 1);
        to1 = clampi(to1, 0, N - 1);
        to2 = clampi(to2, 0, N - 1);
        __syncthreads();
        if (ha != hb) {
#pragma unroll
            for (int x = 0; x < kMaxEPT; ++x) {
                const int32_t e = tid + kThreads * x;
                if (x < a.nx && e < LP) {
                    if (WLDS) {
                        Wl[(int64_t)ha * LP + e] = nwa[x];
                        Wl[(int64_t)hb * LP + e] = nwb[x];
                    } else {
                        Wg[(int64_t)ha * LP + e] = nwa[x];
                        Wg[(int64_t)hb * LP + e] = nwb[x];
                    }
                }
            }
        }
        if (tid == 0) {
            cell_of[i] = c2;
            if (j >= 0) cell_of[j] = c1;
            T[c1] = nT1;
            Q[c1] = nQ1;
            T[c2] = nT2;
            Q[c2] = nQ2;
        }
        if (!reloc) {
            pool_move(pool, pos_i, to1, j);
            pool_move(pool, pos_j, to2, i);
        } else {
            pool_move(pool, pos_i, to1, i);
            if (c1 < c2) {
                for (int32_t c = c1 + 1 + tid; c <= c2; c += kThreads) start[c] -= 1;
            } else {
                for (int32_t c = c2 + 1 + tid; c <= c1; c += kThreads) start[c] += 1;
            }
        }
        __syncthreads();
#pragma unroll
        for (int x = 0; x < kMaxJPL; ++x) {
            const int h = x * kWave + lane;
            if (h == ha) {
                Jr[x] = Ja;
                Ar[x] = Aa;
            } else if (h == hb) {
                Jr[x] = Jb;
                Ar[x] = Ab;
            }
        }
        Ur = Un;
        s0 = n0;
        s1 = n1;
        s2 = n2;
        e_cur = e_new;
        if (lex_less(s0, s1, s2, b0, b1, b2)) {
            b0 = s0;
            b1 = s1;
            b2 = s2;
            best_is_start = 0;
            int32_t *bl = a.best + (int64_t)m * N;
            for (int32_t x = tid; x < N; x += kThreads) bl[x] = cell_of[x];
        }
    }
    // Epilogue: terminal W, J, A and the member's results.
    if (WLDS) {
        for (int64_t h = 0; h < RG; ++h)
            for (int x = 0; x < a.nx; ++x) {
                const int32_t e = tid + kThreads * x;
                if (e < LP) Wg[h * LP + e] = Wl[h * LP + e];
            }
    }
    if (wv == 0) {
#pragma unroll
        for (int x = 0; x < kMaxJPL; ++x) {
            const int h = x * kWave + lane;
            if (h < RG) {
                at<int64_t>(dst, a.off.J)[h] = Jr[x];
                at<int64_t>(dst, a.off.A)[h] = Ar[x];
            }
        }
    }
    if (tid == 0) {
        int64_t *res = a.results + (int64_t)m * kRes;
        res[0] = s0; res[1] = s1; res[2] = s2;
        res[3] = b0; res[4] = b1; res[5] = b2;
        res[6] = n_acc; res[7] = n_eval;
        res[8] = best_is_start;
        res[9] = par;
    }
}

// Building the member slabs from the start layouts.  Identical layouts are
// built once: k_layout_hash hashes every layout (an order-free sum of a
// 64-bit mix of (sample, cell)), k_leader finds for each member the first
// member with an equal layout (hash match confirmed element by element),
// and only those leaders are built; duplicates copy the leader's slab.
__device__ inline uint64_t mix64(uint64_t z) {
    z += 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__global__ void __launch_bounds__(kThreads) k_layout_hash(const int32_t *layouts, int32_t N, uint64_t *hash) {
    __shared__ uint64_t part[kThreads / kWave];
    const int m = blockIdx.x;
    const int32_t *lay = layouts + (int64_t)m * N;
    uint64_t h = 0;
    for (int32_t i = threadIdx.x; i < N; i += kThreads)
        h += mix64(((uint64_t)(uint32_t)i << 32) | (uint32_t)lay[i]);
    h = (uint64_t)wave_sum((int64_t)h);
    if (lane_id() == 0) part[wave_id()] = h;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t t = 0;
        for (int w = 0; w < kThreads / kWave; ++w) t += part[w];
        hash[m] = t;
    }
}

__global__ void __launch_bounds__(64) k_leader(const int32_t *layouts, int32_t N, const uint64_t *hash,
                                               int32_t *leader) {
    const int m = blockIdx.x, lane = lane_id();
    const int32_t *lay = layouts + (int64_t)m * N;
    int32_t found = m;
    for (int u = 0; u < m; ++u) {
        if (hash[u] != hash[m]) continue;
        const int32_t *o = layouts + (int64_t)u * N;
        bool diff = false;
        for (int32_t i = lane; i < N; i += kWave) diff |= (o[i] != lay[i]);
        if (!__ballot(diff)) {
            found = u;
            break;
        }
    }
    if (lane == 0) leader[m] = found;
}

// Cell statistics, validation, start offsets and the sorted member pool of
// every leader.  status gets bit 0 for a cell id out of range, bit 1 for a
// cell over capacity, bit 2 for an empty cell.
__global__ void __launch_bounds__(kThreads) k_build_cells(AnnealArgs a, const int32_t *layouts,
                                                          const int32_t *leader, int32_t *status) {
    extern __shared__ char smem[];
    const int tid = threadIdx.x, lane = lane_id(), wv = wave_id();
    const int m = blockIdx.x;
    if (leader[m] != m) return;
    const int32_t N = a.N, B = a.B;
    char *dst = a.dst + (int64_t)m * a.off.bytes;
    int64_t *cT = reinterpret_cast<int64_t *>(smem);  // [B]
    int64_t *cQ = cT + B;                              // [B]
    int32_t *cN = reinterpret_cast<int32_t *>(cQ + B);  // [B]
    int32_t *off = cN + B;                              // [B]
    int32_t *chunk = off + B;                           // [256]
    int32_t *flag = chunk + kThreads;                   // [1]
    int64_t *red = reinterpret_cast<int64_t *>(((uintptr_t)(flag + 1) + 7) & ~(uintptr_t)7);  // [4]
    const int32_t *lay = layouts + (int64_t)m * N;
    int32_t *cell_of = at<int32_t>(dst, a.off.cell);
    int32_t *pool = at<int32_t>(dst, a.off.pool);
    int32_t *start = at<int32_t>(dst, a.off.start);
    int64_t *T = at<int64_t>(dst, a.off.T);
    int64_t *Q = at<int64_t>(dst, a.off.Q);

    for (int32_t c = tid; c < B; c += kThreads) {
        cT[c] = 0;
        cQ[c] = 0;
        cN[c] = 0;
    }
    if (tid == 0) *flag = 0;
    __syncthreads();
    for (int32_t i = tid; i < N; i += kThreads) {
        const int32_t c = lay[i];
        cell_of[i] = c;
        if (c < 0 || c >= B) {
            atomicOr(flag, 1);
            continue;
        }
        const int64_t ti = a.t[i];
        atomicAdd(reinterpret_cast<unsigned long long *>(&cT[c]), (unsigned long long)ti);
        atomicAdd(reinterpret_cast<unsigned long long *>(&cQ[c]), (unsigned long long)(ti * ti));
        atomicAdd(&cN[c], 1);
    }
    __syncthreads();
    for (int32_t c = tid; c < B; c += kThreads) {
        if (cT[c] > a.C) atomicOr(flag, 2);
        if (cN[c] == 0) atomicOr(flag, 4);
        T[c] = cT[c];
        Q[c] = cQ[c];
    }
    __syncthreads();
    const int32_t st = *flag;
    if (tid == 0) status[m] = st;
    if (st & 1) return;  // uniform
    // start = exclusive prefix of the cell counts (thread-contiguous chunks).
    {
        const int32_t per = (B + kThreads - 1) / kThreads;
        const int32_t lo = tid * per, hi = lo + per < B ? lo + per : B;
        int64_t sum = 0;
        for (int32_t c = lo; c < hi; ++c) sum += cN[c];
        const int64_t incl = wave_incl_scan(sum);
        if (lane == kWave - 1) red[wv] = incl;
        __syncthreads();
        int64_t base = incl - sum;
        for (int w = 0; w < wv; ++w) base += red[w];
        for (int32_t c = lo; c < hi; ++c) {
            start[c] = (int32_t)base;
            off[c] = (int32_t)base;
            base += cN[c];
        }
        if (tid == 0) start[B] = N;
        __syncthreads();
    }
    // pool: ids in ascending order within each cell (stable counting sort).
    for (int32_t base = 0; base < N; base += kThreads) {
        const int32_t i = base + tid;
        chunk[tid] = i < N ? lay[i] : -1;
        __syncthreads();
        int32_t c = -1, rank = 0, tot = 0;
        if (i < N) {
            c = chunk[tid];
            for (int u = 0; u < kThreads; ++u) {
                const int32_t cu = chunk[u];
                tot += (cu == c);
                rank += (cu == c) && (u < tid);
            }
            pool[off[c] + rank] = i;
        }
        __syncthreads();  // every read of off[] for this chunk is done
        if (i < N && rank == tot - 1) off[c] += tot;
        __syncthreads();
    }
}

// W row, A and J of row-shard h of leader m (grid: members x row-shards).
__global__ void __launch_bounds__(kThreads) k_build_rows(AnnealArgs a, const int32_t *leader,
                                                         const int32_t *status) {
    __shared__ int64_t red[kThreads / kWave];
    const int tid = threadIdx.x, lane = lane_id(), wv = wave_id();
    const int64_t m = blockIdx.x / a.RG;
    const int32_t h = (int32_t)(blockIdx.x % a.RG);
    if (leader[m] != m || status[m] != 0) return;
    const int32_t LP = a.LP, D = a.D, G = a.G;
    char *dst = a.dst + m * a.off.bytes;
    const int32_t *pool = at<int32_t>(dst, a.off.pool);
    const int32_t *start = at<int32_t>(dst, a.off.start);
    const int64_t *T = at<int64_t>(dst, a.off.T);
    const int64_t *Q = at<int64_t>(dst, a.off.Q);
    int32_t *W = at<int32_t>(dst, a.off.W);
    const int32_t r = h / G, g = h % G;
    int32_t acc[kMaxEPT];
#pragma unroll
    for (int x = 0; x < kMaxEPT; ++x) acc[x] = 0;
    for (int32_t xs = 0; xs < a.count[g]; ++xs) {
        const int32_t c = r * D + a.slots[g * D + xs];
        for (int32_t pp = start[c]; pp < start[c + 1]; ++pp) {
            const int32_t *qi = a.q + (int64_t)pool[pp] * LP;
#pragma unroll
            for (int x = 0; x < kMaxEPT; ++x) {
                const int32_t e = tid + kThreads * x;
                if (x < a.nx && e < LP) acc[x] += qi[e];
            }
        }
    }
    int64_t esum = 0;
#pragma unroll
    for (int x = 0; x < kMaxEPT; ++x) {
        if (x < a.nx) {
            const int32_t e = tid + kThreads * x;
            const int32_t v = e < LP ? acc[x] : INT32_MIN;
            if (e < LP) W[(int64_t)h * LP + e] = v;
            const int32_t mx = seg_max32(v, a.P);
            if (e < LP && (lane & (a.P - 1)) == 0) esum += mx;
        }
    }
    esum = wave_sum(esum);
    if (lane == 0) red[wv] = esum;
    __syncthreads();
    if (wv == 0) {
        int64_t e = 0;
        for (int w = 0; w < kThreads / kWave; ++w) e += red[w];
        const int64_t A = attention_rs(a, T, Q, r, g, -1, 0, 0, -1, 0, 0);
        if (lane == 0) {
            at<int64_t>(dst, a.off.J)[h] = A + (e << a.F);
            at<int64_t>(dst, a.off.A)[h] = A;
        }
    }
}

// Duplicates copy their leader's slab; every member's score goes to
// results[m][0..2] (and the trajectory-best fields, for the incumbent).
__global__ void __launch_bounds__(kThreads) k_build_final(AnnealArgs a, const int32_t *leader,
                                                          int32_t *status) {
    const int m = blockIdx.x, lane = lane_id();
    const int ld = leader[m];
    char *dst = a.dst + (int64_t)m * a.off.bytes;
    if (ld != m) {
        const int4 *src = reinterpret_cast<const int4 *>(a.dst + (int64_t)ld * a.off.bytes);
        int4 *d4 = reinterpret_cast<int4 *>(dst);
        for (int64_t x = threadIdx.x; x < a.off.bytes / 16; x += kThreads) d4[x] = src[x];
        if (threadIdx.x == 0) status[m] = status[ld];
    }
    if (threadIdx.x >= kWave) return;
    const int32_t st = ld != m ? status[ld] : status[m];
    if (st != 0) return;
    const char *slab = a.dst + (int64_t)ld * a.off.bytes;
    const int64_t *J = reinterpret_cast<const int64_t *>(slab + a.off.J);
    int64_t U = 0;
    if (lane < a.G)
        for (int r = 0; r < a.R; ++r) U += J[(int64_t)r * a.G + lane];
    int64_t jmax = LLONG_MIN;
    for (int h = lane; h < a.RG; h += kWave) jmax = J[h] > jmax ? J[h] : jmax;
    const int64_t s0 = wave_max(lane < a.G ? U : LLONG_MIN);
    const int64_t s1 = wave_sum(lane < a.G ? U : 0);
    const int64_t s2 = wave_max(jmax);
    if (lane == 0) {
        int64_t *res = a.results + (int64_t)m * kRes;
        res[0] = s0; res[1] = s1; res[2] = s2;
        res[3] = s0; res[4] = s1; res[5] = s2;
        res[6] = 0; res[7] = 0; res[8] = 1; res[9] = m;
    }
}

struct LevelEndArgs {
    int32_t pop, N;
    const int64_t *results;   // [pop][kRes]
    const int32_t *best;      // [pop][N]
    const char *src_slabs;    // slabs the level started from
    int64_t slab_bytes, off_cell;
    const int32_t *start_layouts;  // alternative start layouts [pop][N] (first build) or null
    int32_t *xstar;           // [N]
    int64_t *xscore;          // [3]
    int64_t *trace;           // [pop][8] for this level or null
    int32_t *parents_out;     // [pop] for this level or null
    int32_t *next_parent;     // [pop] parents for the next level
    int32_t resample;
    double t_cur, t_next, scale;
    uint64_t seed;
    int32_t level;
    int32_t init_mode;        // 1: x* := lowest-index argmin of results[.][0..2] (no comparison)
    // in-place slabs: slab of each member now and after resampling, and the
    // copies that give duplicated parents' extra children their state
    const int32_t *slab_cur;  // [pop] or null (double-buffered slabs)
    int32_t *slab_next;       // [pop]
    int32_t *copy_src, *copy_dst, *n_copies;  // [pop], [pop], [1]
    int32_t stage_lds;        // hand-over bookkeeping in dynamic LDS (3 pop int32)
};

// After a level: the incumbent update (strict lexicographic improvement,
// ascending member order), the trace, and systematic resampling of the
// terminal states with quantised Boltzmann weights.  One workgroup.
__global__ void __launch_bounds__(1024) k_level_end(LevelEndArgs a) {
    extern __shared__ int32_t lend_par[];  // [3 pop] when a.stage_lds: parents, flags, freed slabs
    __shared__ int64_t sk[16][4];
    __shared__ uint64_t su[16];
    __shared__ double sd[16];
    __shared__ int32_t win;
    const int tid = threadIdx.x, lane = lane_id(), wv = wave_id();
    const int nw = blockDim.x / kWave;
    // 1. argmin over trajectory bests (lowest index on ties).
    int64_t k0 = LLONG_MAX, k1 = LLONG_MAX, k2 = LLONG_MAX, kj = LLONG_MAX;
    const int bo = a.init_mode ? 0 : 3;
    for (int j = tid; j < a.pop; j += blockDim.x) {
        const int64_t *r = a.results + (int64_t)j * kRes + bo;
        if (lex_less(r[0], r[1], r[2], k0, k1, k2) ||
            (r[0] == k0 && r[1] == k1 && r[2] == k2 && j < kj)) {
            k0 = r[0]; k1 = r[1]; k2 = r[2]; kj = j;
        }
    }
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        const int64_t o0 = __shfl_xor(k0, d, kWave), o1 = __shfl_xor(k1, d, kWave);
        const int64_t o2 = __shfl_xor(k2, d, kWave), oj = __shfl_xor(kj, d, kWave);
        if (lex_less(o0, o1, o2, k0, k1, k2) || (o0 == k0 && o1 == k1 && o2 == k2 && oj < kj)) {
            k0 = o0; k1 = o1; k2 = o2; kj = oj;
        }
    }
    if (lane == 0) {
        sk[wv][0] = k0; sk[wv][1] = k1; sk[wv][2] = k2; sk[wv][3] = kj;
    }
    __syncthreads();
    if (tid == 0) {
        for (int w = 1; w < nw; ++w)
            if (lex_less(sk[w][0], sk[w][1], sk[w][2], sk[0][0], sk[0][1], sk[0][2]) ||
                (sk[w][0] == sk[0][0] && sk[w][1] == sk[0][1] && sk[w][2] == sk[0][2] && sk[w][3] < sk[0][3])) {
                for (int f = 0; f < 4; ++f) sk[0][f] = sk[w][f];
            }
        const bool better = a.init_mode ||
                            lex_less(sk[0][0], sk[0][1], sk[0][2], a.xscore[0], a.xscore[1], a.xscore[2]);
        win = better ? (int32_t)sk[0][3] : -1;
        if (better) {
            a.xscore[0] = sk[0][0];
            a.xscore[1] = sk[0][1];
            a.xscore[2] = sk[0][2];
        }
    }
    __syncthreads();
    if (win >= 0) {
        const int64_t *r = a.results + (int64_t)win * kRes;
        const int32_t *srcl;
        if (a.init_mode || r[8]) {
            srcl = a.start_layouts ? a.start_layouts + (int64_t)win * a.N
                                   : reinterpret_cast<const int32_t *>(a.src_slabs + r[9] * a.slab_bytes + a.off_cell);
        } else {
            srcl = a.best + (int64_t)win * a.N;
        }
        for (int x = tid; x < a.N; x += blockDim.x) a.xstar[x] = srcl[x];
    }
    if (a.init_mode) return;
    // 2. trace
    if (a.trace)
        for (int j = tid; j < a.pop; j += blockDim.x)
            for (int f = 0; f < 8; ++f) a.trace[(int64_t)j * 8 + f] = a.results[(int64_t)j * kRes + f];
    // 3. resampling
    if (!a.resample) {
        for (int j = tid; j < a.pop; j += blockDim.x) {
            if (a.parents_out) a.parents_out[j] = -1;
            a.next_parent[j] = j;
            if (a.slab_cur) a.slab_next[j] = a.slab_cur[j];
        }
        if (a.slab_cur && tid == 0) *a.n_copies = 0;
        return;
    }
    double emin = __builtin_inf();
    for (int j = tid; j < a.pop; j += blockDim.x) {
        const int64_t *r = a.results + (int64_t)j * kRes;
        const double e = energy(r[0], r[1], r[2], a.scale);
        emin = e < emin ? e : emin;
    }
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        const double o = __shfl_xor(emin, d, kWave);
        emin = o < emin ? o : emin;
    }
    if (lane == 0) sd[wv] = emin;
    __syncthreads();
    emin = sd[0];
    for (int w = 1; w < nw; ++w) emin = sd[w] < emin ? sd[w] : emin;
    const double den = fabs(emin) > 1.0 ? fabs(emin) : 1.0;
    const double cfac = (1.0 / a.t_next) - (1.0 / a.t_cur);
    // thread-contiguous chunks for an exact uint64 inclusive scan
    const int per = (a.pop + (int)blockDim.x - 1) / (int)blockDim.x;
    const int lo = tid * per, hi = lo + per < a.pop ? lo + per : a.pop;
    uint64_t local = 0;
    for (int j = lo; j < hi; ++j) {
        const int64_t *r = a.results + (int64_t)j * kRes;
        const double en = (energy(r[0], r[1], r[2], a.scale) - emin) / den;
        const double wh = exp_det(-(cfac * en));
        local += (uint64_t)floor(__builtin_ldexp(wh, 40));
    }
    const uint64_t incl = wave_incl_scan_u(local);
    if (lane == kWave - 1) su[wv] = incl;
    __syncthreads();
    uint64_t base = incl - local;
    for (int w = 0; w < wv; ++w) base += su[w];
    uint64_t total = 0;
    for (int w = 0; w < nw; ++w) total += su[w];
    // F_j written to the trace-free scratch: reuse next_parent as staging is
    // not possible (int32), so keep the prefix in the results column 9 of a
    // private copy: recompute per lookup instead (binary search over chunks).
    // Write F into shared per-thread boundaries and do the lookup from them.
    __shared__ uint64_t chunk_lo[1024];
    chunk_lo[tid] = base;
    __syncthreads();
    const U64x4 blk = philox4x64_10(0, (uint64_t)(uint32_t)a.level, 0xFFFFFFFFull, 2, a.seed, 0);
    const uint64_t V = blk.v[0] >> 32;
    const uint64_t P = (uint64_t)a.pop;
    for (int mm = tid; mm < a.pop; mm += blockDim.x) {
        const unsigned __int128 rhs = (unsigned __int128)total * (V + ((uint64_t)mm << 32));
        // F_j * P * 2^32 >= rhs, F nondecreasing: find the first chunk whose
        // end prefix satisfies it, then scan inside the chunk.
        int lo_t = 0, hi_t = (int)blockDim.x - 1;
        // chunk t covers [t*per, min((t+1)*per, pop)); its end prefix is chunk_lo[t+1] (or total)
        while (lo_t < hi_t) {
            const int mid = (lo_t + hi_t) / 2;
            const uint64_t endp = (mid + 1 < (int)blockDim.x) ? chunk_lo[mid + 1] : total;
            if ((unsigned __int128)endp * P * ((uint64_t)1 << 32) >= rhs) hi_t = mid;
            else lo_t = mid + 1;
        }
        uint64_t F = chunk_lo[lo_t];
        int j = lo_t * per;
        int jend = j + per < a.pop ? j + per : a.pop;
        int chosen = a.pop - 1;
        for (; j < jend; ++j) {
            const int64_t *r = a.results + (int64_t)j * kRes;
            const double en = (energy(r[0], r[1], r[2], a.scale) - emin) / den;
            F += (uint64_t)floor(__builtin_ldexp(exp_det(-(cfac * en)), 40));
            if ((unsigned __int128)F * P * ((uint64_t)1 << 32) >= rhs) {
                chosen = j;
                break;
            }
        }
        a.next_parent[mm] = chosen;
        if (a.parents_out) a.parents_out[mm] = chosen;
        if (a.stage_lds) lend_par[mm] = chosen;
    }
    if (!a.slab_cur) return;
    // Slab hand-over: parents are non-decreasing in m.  The first child of a
    // parent takes over its slab; every further child takes the slab of a
    // member without children (ascending order) after a copy.
    __syncthreads();
    if (a.stage_lds) {
        // Parents, has-child flags and the freed slabs in LDS: every test is O(1).
        int32_t *flag = lend_par + a.pop, *freed = flag + a.pop;
        for (int j = tid; j < a.pop; j += blockDim.x) flag[j] = 0;
        __syncthreads();
        for (int mm = tid; mm < a.pop; mm += blockDim.x) flag[lend_par[mm]] = 1;
        __syncthreads();
        int32_t n_dead = 0, n_dup = 0;
        for (int j = lo; j < hi; ++j) {
            n_dead += flag[j] == 0;
            n_dup += (j > 0 && lend_par[j] == lend_par[j - 1]);
        }
        __shared__ int32_t tdead[16], tdupw[16];
        const int32_t idead = (int32_t)wave_incl_scan(n_dead), idup = (int32_t)wave_incl_scan(n_dup);
        if (lane == kWave - 1) {
            tdead[wv] = idead;
            tdupw[wv] = idup;
        }
        __syncthreads();
        int32_t rdead = idead - n_dead, rdup = idup - n_dup, tdup = 0;
        for (int w = 0; w < wv; ++w) {
            rdead += tdead[w];
            rdup += tdupw[w];
        }
        for (int w = 0; w < nw; ++w) tdup += tdupw[w];
        for (int j = lo; j < hi; ++j)
            if (flag[j] == 0) {
                const int32_t sl = a.slab_cur[j];
                freed[rdead] = sl;
                a.copy_dst[rdead] = sl;
                ++rdead;
            }
        __syncthreads();
        for (int m2 = lo; m2 < hi; ++m2) {
            const int32_t p2 = lend_par[m2];
            if (m2 == 0 || p2 != lend_par[m2 - 1]) {
                a.slab_next[m2] = a.slab_cur[p2];
            } else {
                a.slab_next[m2] = freed[rdup];
                a.copy_src[rdup] = a.slab_cur[p2];
                ++rdup;
            }
        }
        if (tid == 0) *a.n_copies = tdup;
        return;
    }
    const int32_t *par = a.next_parent;
    int32_t n_dead = 0, n_dup = 0;
    for (int j = lo; j < hi; ++j) {
        int32_t l = 0, h = a.pop;  // lower bound of j in par
        while (l < h) {
            const int32_t md = (l + h) >> 1;
            if (par[md] < j) l = md + 1;
            else h = md;
        }
        n_dead += !(l < a.pop && par[l] == j);
        n_dup += (j > 0 && par[j] == par[j - 1]);
    }
    __shared__ int32_t sdead[16], sdup[16];
    const int32_t idead = (int32_t)wave_incl_scan(n_dead), idup = (int32_t)wave_incl_scan(n_dup);
    if (lane == kWave - 1) {
        sdead[wv] = idead;
        sdup[wv] = idup;
    }
    __syncthreads();
    int32_t rdead = idead - n_dead, rdup = idup - n_dup, tdup = 0;
    for (int w = 0; w < wv; ++w) {
        rdead += sdead[w];
        rdup += sdup[w];
    }
    for (int w = 0; w < nw; ++w) tdup += sdup[w];
    for (int j = lo; j < hi; ++j) {
        int32_t l = 0, h = a.pop;
        while (l < h) {
            const int32_t md = (l + h) >> 1;
            if (par[md] < j) l = md + 1;
            else h = md;
        }
        if (!(l < a.pop && par[l] == j)) a.copy_dst[rdead++] = a.slab_cur[j];
    }
    __syncthreads();
    for (int m2 = lo; m2 < hi; ++m2) {
        if (m2 == 0 || par[m2] != par[m2 - 1]) {
            a.slab_next[m2] = a.slab_cur[par[m2]];
        } else {
            a.slab_next[m2] = a.copy_dst[rdup];
            a.copy_src[rdup] = a.slab_cur[par[m2]];
            ++rdup;
        }
    }
    if (tid == 0) *a.n_copies = tdup;
}

// population[m] = cell_of of slab parent[m] (or m).
// Population rows from the slabs (member m from slab parent[m]).  With
// err set (a wait of the whole-schedule kernel gave up, so the slab map may
// be unwritten) it copies nothing.
__global__ void k_gather_population(const char *slabs, int64_t slab_bytes, int64_t off_cell,
                                    const int32_t *parent, int32_t N, int32_t *population,
                                    const int32_t *err) {
    if (err && *err) return;
    const int m = blockIdx.x;
    const int par = parent ? parent[m] : m;
    const int32_t *src = reinterpret_cast<const int32_t *>(slabs + (int64_t)par * slab_bytes + off_cell);
    for (int x = threadIdx.x; x < N; x += blockDim.x) population[(int64_t)m * N + x] = src[x];
}

__global__ void k_compare_score(const int64_t *a, const int64_t *b, const int32_t *status, int32_t *out) {
    if (threadIdx.x == 0) *out = (status[0] == 0 && a[0] == b[0] && a[1] == b[1] && a[2] == b[2]) ? 1 : 0;
}

static int64_t align_up(int64_t x) { return (x + 255) & ~(int64_t)255; }

// Polls before a wait of the whole-schedule kernel gives up: 2^22 (seconds
// of waiting), or ROUTEPACK_WAIT_SPINS (at least 32) when that is set.
static unsigned wait_spin_limit() {
    const char *v = getenv("ROUTEPACK_WAIT_SPINS");
    if (!v || !*v) return 1u << 22;
    const unsigned long x = strtoul(v, nullptr, 10);
    return x < 32 ? 32u : (x > (1ul << 30) ? (1u << 30) : (unsigned)x);
}

static SlabOffsets slab_layout(int64_t N, int64_t B, int64_t RG, int64_t LP) {
    SlabOffsets o;
    int64_t p = 0;
    o.cell = p; p = align_up(p + 4 * N);
    o.pool = p; p = align_up(p + 4 * N);
    o.start = p; p = align_up(p + 4 * (B + 1));
    o.T = p; p = align_up(p + 8 * B);
    o.Q = p; p = align_up(p + 8 * B);
    o.W = p; p = align_up(p + 4 * RG * LP);
    o.J = p; p = align_up(p + 8 * RG);
    o.A = p; p = align_up(p + 8 * RG);
    o.bytes = p;
    return o;
}

}  // namespace rp

using namespace rp;

extern "C" int routepack_anneal(const routepack_problem *prob, const int32_t *lengths,
                                const int32_t *q, int32_t n_rows, int32_t pop_size,
                                int32_t *population, const routepack_anneal_params *prm,
                                int32_t *best_layout, int64_t *best_score, int64_t *trace,
                                int32_t *parents, uint8_t *step_log, hipStream_t stream) {
    Topology topo;
    RP_TRY(check_problem(prob, &topo));
    if (!prm || !lengths || !population || !best_layout || !best_score) return ROUTEPACK_E_INVALID;
    if (prob->n_layers > 0 && !q) return ROUTEPACK_E_INVALID;
    if (n_rows < 1 || pop_size < 1 || prm->n_sweeps < 0 || prm->steps_per_sweep < 0)
        return ROUTEPACK_E_INVALID;
    if (prm->n_sweeps > 0 && !prm->temperatures) return ROUTEPACK_E_INVALID;
    for (int n = 0; n < prm->n_sweeps; ++n) {
        if (!(prm->temperatures[n] > 0.0)) return ROUTEPACK_E_INVALID;
        if (n > 0 && !(prm->temperatures[n] < prm->temperatures[n - 1])) return ROUTEPACK_E_INVALID;
    }
    if (prm->n_sweeps > 0 && prm->t_next > 0.0 &&
        !(prm->t_next < prm->temperatures[prm->n_sweeps - 1]))
        return ROUTEPACK_E_INVALID;
    const int32_t N = prob->n_samples, L = prob->n_layers, P = prob->n_ranks;
    const int32_t D = topo.D, G = topo.G;
    const int64_t B64 = (int64_t)n_rows * D, RG64 = (int64_t)n_rows * G, LP64 = (int64_t)L * P;
    if (B64 > N) return ROUTEPACK_E_LAYOUT;  // a feasible layout needs N >= R*D
    if ((P & (P - 1)) != 0 || P > 64 || LP64 > (int64_t)kThreads * kMaxEPT ||
        RG64 > (int64_t)kWave * kMaxJPL || G > 64 || topo.max_count > 64 ||
        prob->n_stages > kMaxStages)
        return ROUTEPACK_E_UNSUPPORTED;
    WindowStats ws;
    RP_TRY(window_stats(prob, lengths, q, &ws, stream));
    if (ws.min_t < 1 || ws.q_negative) return ROUTEPACK_E_INVALID;
    RP_TRY(overflow_check(prob, n_rows, ws, true));

    Scratch scr(stream);
    DeviceProblem dp;
    RP_TRY(upload_problem(prob, topo, scr, &dp, stream));
    const SlabOffsets off = slab_layout(N, B64, RG64, LP64);
    char *slabA = scr.get<char>((size_t)pop_size * off.bytes);
    int32_t *best = scr.get<int32_t>((size_t)pop_size * N);
    int64_t *results = scr.get<int64_t>((size_t)pop_size * kRes);
    int32_t *status = scr.get<int32_t>(pop_size + 1);
    int32_t *parent = scr.get<int32_t>(pop_size);
    int64_t *chk_score = scr.get<int64_t>(3);
    int32_t *chk = scr.get<int32_t>(2);
    int64_t *xscore_in = scr.get<int64_t>(3);
    int32_t *qzero = scr.get<int32_t>(LP64 > 0 ? LP64 : 1);
    if (scr.failed()) return ROUTEPACK_E_DEVICE;
    RP_HIP(hipMemsetAsync(qzero, 0, sizeof(int32_t) * (LP64 > 0 ? LP64 : 1), stream));

    AnnealArgs a;
    memset(&a, 0, sizeof(a));
    a.t = lengths; a.q = q;
    a.N = N; a.L = L; a.P = P; a.D = D; a.G = G; a.R = n_rows; a.S = prob->n_stages;
    a.F = prob->frac_bits; a.K = prm->steps_per_sweep;
    a.LP = (int32_t)LP64; a.RG = (int32_t)RG64; a.B = (int32_t)B64;
    a.nx = (int32_t)((LP64 + kThreads - 1) / kThreads);
    a.pshift = 0;
    while ((1 << a.pshift) < P) ++a.pshift;
    a.C = prob->capacity;
    a.scale = ldexp((double)prob->capacity, prob->frac_bits);
    {
        int e2 = 0;
        a.scale_pow2 = frexp(a.scale, &e2) == 0.5 ? 1 : 0;
        a.inv_scale = a.scale_pow2 ? ldexp(1.0, 1 - e2) : 0.0;
    }
    for (int s = 0; s < prob->n_stages; ++s) {
        a.alpha[s] = prob->alpha_fp[s];
        a.beta[s] = prob->beta_fp[s];
    }
    a.slots = dp.slots; a.count = dp.count; a.slot_shard = dp.slot_shard;
    a.qzero = qzero;
    a.sum32 = (long double)L * (long double)w_entry_bound(prob, ws) < 2147483648.0L ? 1 : 0;
    a.off = off;
    a.best = best; a.results = results;
    a.seed = prm->seed; a.p_guide = prm->p_guide_u32; a.rho = prm->rho_u32;

    // Build member slabs from the population (each distinct layout once) and
    // validate them.
    a.dst = slabA;
    uint64_t *hash = scr.get<uint64_t>(pop_size);
    int32_t *leader = scr.get<int32_t>(pop_size);
    if (scr.failed()) return ROUTEPACK_E_DEVICE;
    const size_t lds_build = (size_t)B64 * 24 + kThreads * 4 + 4 + 8 + 32 + 8;
    if (lds_build > 160 * 1024) return ROUTEPACK_E_UNSUPPORTED;
    RP_HIP(hipFuncSetAttribute((const void *)k_build_cells, hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)lds_build));
    hipLaunchKernelGGL(k_layout_hash, dim3(pop_size), dim3(kThreads), 0, stream, population, N, hash);
    hipLaunchKernelGGL(k_leader, dim3(pop_size), dim3(64), 0, stream, population, N, hash, leader);
    hipLaunchKernelGGL(k_build_cells, dim3(pop_size), dim3(kThreads), lds_build, stream, a, population,
                       leader, status);
    hipLaunchKernelGGL(k_build_rows, dim3((unsigned)(pop_size * RG64)), dim3(kThreads), 0, stream, a,
                       leader, status);
    hipLaunchKernelGGL(k_build_final, dim3(pop_size), dim3(kThreads), 0, stream, a, leader, status);
    RP_HIP(hipGetLastError());
    std::vector<int32_t> hstat(pop_size);
    RP_HIP(hipMemcpyAsync(hstat.data(), status, sizeof(int32_t) * pop_size, hipMemcpyDeviceToHost, stream));
    RP_HIP(hipStreamSynchronize(stream));
    for (int j = 0; j < pop_size; ++j)
        if (hstat[j]) return ROUTEPACK_E_LAYOUT;

    // Minimum start score (non-regression reference) and the incumbent.
    std::vector<int64_t> hres((size_t)pop_size * kRes);
    RP_HIP(hipMemcpyAsync(hres.data(), results, sizeof(int64_t) * pop_size * kRes,
                          hipMemcpyDeviceToHost, stream));
    int64_t hx[3];
    RP_HIP(hipMemcpyAsync(hx, best_score, sizeof(hx), hipMemcpyDeviceToHost, stream));
    RP_HIP(hipStreamSynchronize(stream));
    int64_t ref[3] = {hres[0], hres[1], hres[2]};
    for (int j = 1; j < pop_size; ++j) {
        const int64_t *r = &hres[(size_t)j * kRes];
        if (lex_less(r[0], r[1], r[2], ref[0], ref[1], ref[2])) {
            ref[0] = r[0]; ref[1] = r[1]; ref[2] = r[2];
        }
    }
    LevelEndArgs le;
    memset(&le, 0, sizeof(le));
    const size_t lend_lds = (size_t)12 * pop_size;
    const bool lend_stage = lend_lds <= 112 * 1024;
    if (lend_stage && lend_lds > 0)
        RP_HIP(hipFuncSetAttribute((const void *)k_level_end, hipFuncAttributeMaxDynamicSharedMemorySize,
                                   (int)lend_lds));
    const size_t lend_shm = lend_stage ? lend_lds : 0;
    le.pop = pop_size; le.N = N; le.results = results; le.best = best;
    le.slab_bytes = off.bytes; le.off_cell = off.cell;
    le.xstar = best_layout; le.xscore = best_score;
    le.scale = a.scale; le.seed = prm->seed; le.next_parent = parent;
    if (prm->init_incumbent) {
        le.init_mode = 1;
        le.start_layouts = population;
        hipLaunchKernelGGL(k_level_end, dim3(1), dim3(1024), lend_shm, stream, le);
        RP_HIP(hipGetLastError());
        le.init_mode = 0;
        le.start_layouts = nullptr;
    } else {
        // The given x* must be feasible and carry its own score.
        RP_TRY(eval_layouts(prob, topo, dp, lengths, q, n_rows, 1, best_layout, chk_score, status,
                            nullptr, nullptr, nullptr, stream));
        hipLaunchKernelGGL(k_compare_score, dim3(1), dim3(64), 0, stream, chk_score, best_score,
                           status, chk);
        int32_t ok = 0;
        RP_HIP(hipMemcpyAsync(&ok, chk, sizeof(ok), hipMemcpyDeviceToHost, stream));
        RP_HIP(hipStreamSynchronize(stream));
        if (!ok) return ROUTEPACK_E_LAYOUT;
        if (lex_less(hx[0], hx[1], hx[2], ref[0], ref[1], ref[2])) {
            ref[0] = hx[0]; ref[1] = hx[1]; ref[2] = hx[2];
        }
    }
    (void)xscore_in;

    // Kernel choice: one wave per member when its state fits LDS (members
    // updated in place, slabs handed over at resampling) -- the chain kernels
    // when the shape fits their lane layout (the whole schedule in one
    // cooperative launch when every workgroup can stay resident, else one
    // launch per level), else the flat wave kernel --, else one workgroup per
    // member over double-buffered slabs.
    // ROUTEPACK_ANNEAL_KERNEL=chain_run|chain|wave|workgroup requests one
    // kernel; a request the problem does not fit fails with
    // ROUTEPACK_E_UNSUPPORTED.
    int32_t mpw = 0, chain_pv = 0, chain_dv = 0;
    bool tlds = false;
    const char *force = getenv("ROUTEPACK_ANNEAL_KERNEL");
    const bool want_run = !force || strcmp(force, "chain_run") == 0;
    const bool want_chain = !force || strcmp(force, "chain") == 0;
    const bool want_wave = !force || strcmp(force, "wave") == 0;
    const bool want_group = !force || strcmp(force, "workgroup") == 0;
    if (!want_run && !want_chain && !want_wave && !want_group) return ROUTEPACK_E_INVALID;
    a.pop = pop_size;
    int dev = 0, n_cu = 256, coop = 0;
    RP_HIP(hipGetDevice(&dev));
    RP_HIP(hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev));
    RP_HIP(hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev));
    const bool chain_fits = (want_run || want_chain) && chain_plan(a, n_cu, topo.max_count, &chain_pv, &chain_dv);
    RunArgs run;
    memset(&run, 0, sizeof(run));
    bool whole = false;
    if (chain_fits && want_run && coop && prm->n_sweeps > 0) {
        const int rc = chain_run(a, run, chain_pv, chain_dv, n_cu, false, stream);
        if (rc != ROUTEPACK_OK && rc != ROUTEPACK_E_UNSUPPORTED) return rc;
        whole = rc == ROUTEPACK_OK;
    }
    const bool chain = chain_fits && !whole && want_chain;
    if (whole || chain) {
        a.slabs = slabA;
        int32_t *qt = scr.get<int32_t>(LP64 > 0 ? (size_t)N * LP64 : 1);
        if (scr.failed()) return ROUTEPACK_E_DEVICE;
        RP_TRY(chain_prepare(a, qt, stream));
        if (a.hq) {  // (64 ranks: the members' cost prefixes live in HBM)
            a.gcp = scr.get<int64_t>((size_t)pop_size * (size_t)a.cp_stride);
            if (scr.failed()) return ROUTEPACK_E_DEVICE;
        }
    }
    const bool fast = whole || chain || (want_wave && wave_plan(a, n_cu, &mpw, &tlds));
    if (!fast && !want_group) return ROUTEPACK_E_UNSUPPORTED;
    if (prm->level_kernel)
        *prm->level_kernel = whole ? ROUTEPACK_KERNEL_CHAIN_RUN
                                   : (chain ? ROUTEPACK_KERNEL_CHAIN
                                            : (fast ? ROUTEPACK_KERNEL_WAVE : ROUTEPACK_KERNEL_WORKGROUP));
    char *slabB = nullptr;
    int32_t *slab_of[2] = {nullptr, nullptr};
    int32_t *copy_src = nullptr, *copy_dst = nullptr, *n_copies = nullptr;
    if (fast) {
        slab_of[0] = scr.get<int32_t>(pop_size);
        slab_of[1] = scr.get<int32_t>(pop_size);
        copy_src = scr.get<int32_t>(pop_size);
        copy_dst = scr.get<int32_t>(pop_size);
        n_copies = scr.get<int32_t>(1);
        if (scr.failed()) return ROUTEPACK_E_DEVICE;
        std::vector<int32_t> iota(pop_size);
        for (int j = 0; j < pop_size; ++j) iota[j] = j;
        RP_HIP(hipMemcpyAsync(slab_of[0], iota.data(), sizeof(int32_t) * pop_size, hipMemcpyHostToDevice,
                              stream));
        RP_HIP(hipStreamSynchronize(stream));  // iota is a host temporary
        a.slabs = slabA;
        a.xscore = best_score;
    } else {
        slabB = scr.get<char>((size_t)pop_size * off.bytes);
        if (scr.failed()) return ROUTEPACK_E_DEVICE;
    }
    const size_t lds_w = (size_t)RG64 * LP64 * 4;
    const bool wlds = 128 + lds_w <= 160 * 1024;
    const size_t lds_level = 128 + (wlds ? lds_w : 0);
    if (!fast && wlds)
        RP_HIP(hipFuncSetAttribute((const void *)k_anneal_level<true>,
                                   hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_level));
    char *src = slabA, *dst = slabB;
    const int32_t *cur_parent = nullptr;
    int cur = 0;
    std::vector<hipEvent_t> ev;
    if (prm->level_kernel_ms) {
        ev.resize(2 * (size_t)prm->n_sweeps);
        for (auto &e : ev) RP_HIP(hipEventCreate(&e));
    }
    struct EventGuard {
        std::vector<hipEvent_t> &v;
        ~EventGuard() { for (auto e : v) (void)hipEventDestroy(e); }
    } ev_guard{ev};
    if (whole) {
        // The whole schedule in one cooperative launch.
        double *temps_d = scr.get<double>(prm->n_sweeps);
        uint32_t *vwords = scr.get<uint32_t>(prm->n_sweeps);
        unsigned *bar = scr.get<unsigned>(2);
        int32_t *slab_final = scr.get<int32_t>(pop_size);
        // by level parity: a workgroup that runs ahead into the next level
        // writes the other half
        double *energy_d = scr.get<double>((size_t)2 * pop_size);
        int64_t *wg_best = scr.get<int64_t>((size_t)8 * pop_size);
        double *wg_emin = scr.get<double>((size_t)2 * pop_size);
        unsigned *flags = scr.get<unsigned>((size_t)2 * pop_size);  // hand-over flags and counts
        const int64_t blob_bytes = run_blob_bytes(a.lds_member);
        char *blobs = scr.get<char>((size_t)pop_size * (size_t)blob_bytes);
        if (scr.failed()) return ROUTEPACK_E_DEVICE;
        RP_HIP(hipMemcpyAsync(temps_d, prm->temperatures, sizeof(double) * prm->n_sweeps, hipMemcpyHostToDevice,
                              stream));
        RP_HIP(hipMemsetAsync(bar, 0, 2 * sizeof(unsigned), stream));
        RP_HIP(hipMemsetAsync(flags, 0, 2 * sizeof(unsigned) * (size_t)pop_size, stream));
        RP_TRY(launch_resample_words(a.seed, prm->sweep_offset, prm->n_sweeps, vwords, stream));
        run.vwords = vwords;
        a.slabs = slabA;
        a.xscore = best_score;
        run.temps = temps_d;
        run.n_sweeps = prm->n_sweeps;
        run.offset = prm->sweep_offset;
        run.t_after = prm->t_next;
        run.trace = trace;
        run.parents_out = parents;
        run.step_log = step_log;
        run.xstar = best_layout;
        run.xscore = best_score;
        run.bar = bar;
        run.err = reinterpret_cast<int32_t *>(bar + 1);
        run.slab_of_out = slab_final;
        run.energy = energy_d;
        run.wg_best = wg_best;
        run.wg_emin = wg_emin;
        run.blobs = blobs;
        run.blob_bytes = blob_bytes;
        run.pub = flags;
        run.got = flags + pop_size;
        run.spin_limit = wait_spin_limit();
        if (a.rv == 2) {  // the two-per-lane variant keeps its level-end tables in HBM
            run.lend_stride = run_lend_bytes(pop_size);
            run.lend = scr.get<char>((size_t)((pop_size + a.mpw - 1) / a.mpw) * (size_t)run.lend_stride);
            if (scr.failed()) return ROUTEPACK_E_DEVICE;
        }
        hipEvent_t e0 = nullptr, e1 = nullptr;
        if (prm->level_kernel_ms) {
            RP_HIP(hipEventCreate(&e0));
            RP_HIP(hipEventCreate(&e1));
            RP_HIP(hipEventRecord(e0, stream));
        }
        const int rc = chain_run(a, run, chain_pv, chain_dv, n_cu, true, stream);
        if (rc != ROUTEPACK_OK) {
            if (e0) (void)hipEventDestroy(e0);
            if (e1) (void)hipEventDestroy(e1);
            return rc;
        }
        if (e1) RP_HIP(hipEventRecord(e1, stream));
        hipLaunchKernelGGL(k_gather_population, dim3(pop_size), dim3(256), 0, stream, slabA, off.bytes, off.cell,
                           slab_final, N, population, (const int32_t *)run.err);
        RP_HIP(hipGetLastError());
        RP_TRY(eval_layouts(prob, topo, dp, lengths, q, n_rows, 1, best_layout, chk_score, status, nullptr,
                            nullptr, nullptr, stream));
        hipLaunchKernelGGL(k_compare_score, dim3(1), dim3(64), 0, stream, chk_score, best_score, status, chk);
        int32_t ok = 0, err = 0;
        RP_HIP(hipMemcpyAsync(&ok, chk, sizeof(ok), hipMemcpyDeviceToHost, stream));
        RP_HIP(hipMemcpyAsync(&err, run.err, sizeof(err), hipMemcpyDeviceToHost, stream));
        RP_HIP(hipMemcpyAsync(hx, best_score, sizeof(hx), hipMemcpyDeviceToHost, stream));
        RP_HIP(hipStreamSynchronize(stream));
        if (e0) {
            float ms = 0.0f;
            const hipError_t et = hipEventElapsedTime(&ms, e0, e1);
            (void)hipEventDestroy(e0);
            (void)hipEventDestroy(e1);
            if (et != hipSuccess) return ROUTEPACK_E_DEVICE;
            // one kernel for every level: each entry gets an equal share
            for (int n = 0; n < prm->n_sweeps; ++n) prm->level_kernel_ms[n] = ms / prm->n_sweeps;
        }
        if (err) return ROUTEPACK_E_DEVICE;
        if (!ok) return ROUTEPACK_E_INTERNAL;
        if (lex_less(ref[0], ref[1], ref[2], hx[0], hx[1], hx[2])) return ROUTEPACK_E_INTERNAL;
        return ROUTEPACK_OK;
    }
    for (int n = 0; n < prm->n_sweeps; ++n) {
        a.level = prm->sweep_offset + n;
        a.temp = prm->temperatures[n];
        a.step_log = step_log ? step_log + (size_t)n * pop_size * a.K : nullptr;
        if (!ev.empty()) RP_HIP(hipEventRecord(ev[2 * n], stream));
        if (fast) {
            a.slab_of = slab_of[cur];
            if (chain) RP_TRY(launch_anneal_chain(a, chain_pv, chain_dv, stream));
            else RP_TRY(launch_anneal_wave(a, tlds, stream));
        } else {
            a.src = src;
            a.dst = dst;
            a.parent = cur_parent;
            if (wlds)
                hipLaunchKernelGGL(k_anneal_level<true>, dim3(pop_size), dim3(kThreads), lds_level, stream, a);
            else
                hipLaunchKernelGGL(k_anneal_level<false>, dim3(pop_size), dim3(kThreads), lds_level, stream, a);
        }
        if (!ev.empty()) RP_HIP(hipEventRecord(ev[2 * n + 1], stream));
        const double t_after = (n + 1 < prm->n_sweeps) ? prm->temperatures[n + 1] : prm->t_next;
        le.src_slabs = src;
        le.trace = trace ? trace + (size_t)n * pop_size * 8 : nullptr;
        le.parents_out = parents ? parents + (size_t)n * pop_size : nullptr;
        le.resample = t_after > 0.0 ? 1 : 0;
        le.t_cur = prm->temperatures[n];
        le.t_next = t_after;
        le.level = a.level;
        le.stage_lds = lend_stage ? 1 : 0;
        if (fast) {
            le.slab_cur = slab_of[cur];
            le.slab_next = slab_of[cur ^ 1];
            le.copy_src = copy_src;
            le.copy_dst = copy_dst;
            le.n_copies = n_copies;
        }
        hipLaunchKernelGGL(k_level_end, dim3(1), dim3(1024), lend_shm, stream, le);
        RP_HIP(hipGetLastError());
        if (fast) {
            RP_TRY(launch_copy_slabs(slabA, off.bytes, copy_src, copy_dst, n_copies, pop_size, stream));
            cur ^= 1;
        } else {
            cur_parent = parent;
            std::swap(src, dst);
        }
    }
    // Output population: start states of the next level.
    if (prm->n_sweeps > 0) {
        if (fast)
            hipLaunchKernelGGL(k_gather_population, dim3(pop_size), dim3(256), 0, stream, slabA, off.bytes,
                               off.cell, slab_of[cur], N, population, (const int32_t *)nullptr);
        else
            hipLaunchKernelGGL(k_gather_population, dim3(pop_size), dim3(256), 0, stream, src, off.bytes,
                               off.cell, cur_parent, N, population, (const int32_t *)nullptr);
    }
    RP_HIP(hipGetLastError());
    // Validate x* and the non-regression guarantee.
    RP_TRY(eval_layouts(prob, topo, dp, lengths, q, n_rows, 1, best_layout, chk_score, status,
                        nullptr, nullptr, nullptr, stream));
    hipLaunchKernelGGL(k_compare_score, dim3(1), dim3(64), 0, stream, chk_score, best_score, status, chk);
    int32_t ok = 0;
    RP_HIP(hipMemcpyAsync(&ok, chk, sizeof(ok), hipMemcpyDeviceToHost, stream));
    RP_HIP(hipMemcpyAsync(hx, best_score, sizeof(hx), hipMemcpyDeviceToHost, stream));
    RP_HIP(hipStreamSynchronize(stream));
    for (int n = 0; n < (int)ev.size() / 2; ++n) {
        float ms = 0.0f;
        RP_HIP(hipEventElapsedTime(&ms, ev[2 * n], ev[2 * n + 1]));
        prm->level_kernel_ms[n] = ms;
    }
    if (!ok) return ROUTEPACK_E_INTERNAL;
    if (lex_less(ref[0], ref[1], ref[2], hx[0], hx[1], hx[2])) return ROUTEPACK_E_INTERNAL;
    return ROUTEPACK_OK;
}
