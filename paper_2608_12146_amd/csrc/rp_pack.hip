// Row-count search, FixedRowFFD and the feasible seed population (Sec. 3.2,
// Sec. 4.1.1, Alg. 2) on gfx950.
//
//  k_rank_sort     sigma = samples ordered by (-t, i): the rank of sample i is
//                  the number of samples that precede it (exact, parallel).
//  k_ffd           FixedRowFFD for K = R*D cells, one wave: the K longest
//                  samples open the cells; every later sample goes to the
//                  lowest-index cell with room, found with a two-level ballot
//                  (per-64-cell maximum room, then the cells of that chunk).
//  k_seed_words    Philox4x64-10 words of every randomized draw, in parallel.
//  k_pack_trials   one wave per candidate: block 0 pairs x_length's cells
//                  with width 1; block b >= 1 runs trial b (WindowShuffle,
//                  RandomizedBestFit, EDPAwarePair with width w).
//  k_canonical     canonical form of every candidate: cells are disjoint, so
//                  ordering the cells of a row-shard by their sorted id tuples
//                  is ordering them by smallest id, and ordering rows by their
//                  tuple of cell tuples is ordering them by the smallest id of
//                  the cell in slot 0.
//  k_pack_select   keep x_length, x_paired (if strictly better), and every
//                  successful trial; drop canonical duplicates (first kept);
//                  order by (score, discovery); fill the population cyclically.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "rp_device.h"
#include "rp_internal.h"

namespace rp {

int eval_layouts(const routepack_problem *p, const Topology &topo, const DeviceProblem &dp,
                 const int32_t *t, const int32_t *q, int32_t R, int64_t n, const int32_t *layouts,
                 int64_t *scores, int32_t *status, int64_t *J, double *diag,
                 const int64_t *rank_load, hipStream_t stream);
__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t v);

constexpr int kMaxCells = 4096;

__global__ void __launch_bounds__(256) k_rank_sort(const int32_t *__restrict__ t, int32_t N,
                                                   int32_t *__restrict__ sigma) {
    __shared__ __align__(16) int32_t tile[1024];
    const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    const int32_t ti = i < N ? t[i] : 0;
    int32_t rank = 0;
    for (int32_t base = 0; base < N; base += 1024) {
        for (int x = threadIdx.x; x < 1024; x += blockDim.x) tile[x] = base + x < N ? t[base + x] : -1;
        __syncthreads();
        const int32_t lim = N - base < 1024 ? N - base : 1024;
        // four lengths per 16-byte LDS read, several reads in flight
        const int4 *t4 = reinterpret_cast<const int4 *>(tile);
        const int32_t lim4 = lim >> 2;
#pragma unroll 4
        for (int x4 = 0; x4 < lim4; ++x4) {
            const int4 v = t4[x4];
            const int32_t x = base + 4 * x4;
            rank += (v.x > ti) || (v.x == ti && x < i);
            rank += (v.y > ti) || (v.y == ti && x + 1 < i);
            rank += (v.z > ti) || (v.z == ti && x + 2 < i);
            rank += (v.w > ti) || (v.w == ti && x + 3 < i);
        }
        for (int x = 4 * lim4; x < lim; ++x) {
            const int32_t tj = tile[x];
            rank += (tj > ti) || (tj == ti && base + x < i);
        }
        __syncthreads();
    }
    if (i < N) sigma[rank] = i;
}

// FixedRowFFD (one wave).  ok = 1 and cell_of filled on success.
__global__ void __launch_bounds__(64) k_ffd(const int32_t *__restrict__ t, const int32_t *__restrict__ sigma,
                                            int32_t N, int64_t C, int32_t K, int32_t *cell_of, int32_t *ok) {
    __shared__ int64_t room[kMaxCells];
    const int lane = lane_id();
    const int nchunk = (K + kWave - 1) / kWave;
    for (int c = lane; c < K; c += kWave) {
        const int32_t i = sigma[c];
        room[c] = C - t[i];
        cell_of[i] = c;
    }
    __syncthreads();
    // lane x holds the largest room of chunk x (cells 64x .. 64x+63)
    int64_t cmax = -1;
    for (int x = 0; x < nchunk; ++x) {
        const int c = x * kWave + lane;
        const int64_t v = wave_max(c < K ? room[c] : -1);
        if (lane == x) cmax = v;
    }
    // Items after the first K: this block's items and lengths (s0, t0), the
    // next block's (s1, t1) and the items of the one after (s2), loaded a
    // block of 64 ahead; item hb + x's cell stays in lane x until its block
    // is stored, so no step waits on memory.  Only this wave touches the
    // LDS rooms, so a wave-level fence orders a step's update before the
    // next step's reads.
    int32_t hb = K;
    const int32_t i0 = hb + lane, i1 = i0 + kWave, i2 = i1 + kWave;
    int32_t s0 = i0 < N ? sigma[i0] : 0, s1 = i1 < N ? sigma[i1] : 0, s2 = i2 < N ? sigma[i2] : 0;
    int32_t t0 = i0 < N ? t[s0] : 0, t1 = i1 < N ? t[s1] : 0;
    int32_t p_item = -1, p_cell = 0;
    int32_t good = 1;
    for (int32_t h = K; h < N; ++h) {
        if (h - hb == kWave) {
            if (p_item >= 0) cell_of[p_item] = p_cell;
            p_item = -1;
            hb += kWave;
            s0 = s1;
            t0 = t1;
            s1 = s2;
            const int32_t j1 = hb + kWave + lane, j2 = j1 + kWave;
            t1 = j1 < N ? t[s1] : 0;
            s2 = j2 < N ? sigma[j2] : 0;
        }
        const int32_t i = __builtin_amdgcn_readlane(s0, h - hb);
        const int64_t ti = __builtin_amdgcn_readlane(t0, h - hb);
        const uint64_t m1 = __ballot(lane < nchunk && cmax >= ti);
        if (!m1) {
            good = 0;
            break;
        }
        const int x = first_lane(m1);
        const int c0 = x * kWave;
        const int64_t r = (c0 + lane < K) ? room[c0 + lane] : -1;
        const int c = c0 + first_lane(__ballot(r >= ti));
        const int64_t nr = (c0 + lane == c) ? r - ti : r;
        if (c0 + lane == c) room[c] = nr;
        const int64_t nm = wave_max(nr);
        if (lane == x) cmax = nm;
        if (lane == h - hb) {
            p_item = i;
            p_cell = c;
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    if (p_item >= 0) cell_of[p_item] = p_cell;
    if (lane == 0) *ok = good;
}

// words[b][0][h] shuffle draws, words[b][1][h] best-fit draws (h < N),
// words[b][2][pos] pairing draws (pos < K), for trial b = 1 .. M-2.
__global__ void k_seed_words(uint64_t seed, int32_t n_trials, int32_t N, int32_t K, uint64_t *words) {
    const int64_t per = 2 * (int64_t)N + K;
    const int64_t total = (int64_t)(n_trials - 2) * per;
    for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < total;
         x += (int64_t)gridDim.x * blockDim.x) {
        const int64_t b = x / per + 1, r = x % per;
        uint64_t draw, phase;
        if (r < N) { draw = r; phase = 0; }
        else if (r < 2 * (int64_t)N) { draw = r - N; phase = 1; }
        else { draw = r - 2 * (int64_t)N; phase = 2; }
        words[(b - 1) * per + r] = philox4x64_10(draw, (uint64_t)b, phase, 3, seed, 0).v[0];
    }
}

struct TrialArgs {
    const int32_t *t, *q, *sigma, *x_length;
    int32_t N, L, P, D, G, R, K, RG, LP, w;
    int64_t C;
    const int32_t *slots, *count;
    const uint64_t *words;   // [M-2][2N+K]
    // per-block scratch
    int32_t *cellk;          // [M-1][N]
    int32_t *Qc;             // [M-1][K][LP]
    int64_t *peak;           // [M-1][K]
    int32_t *order;          // [M-1][K]
    int32_t *Wt;             // [M-1][RG][LP]
    int64_t *base, *after, *pkv;  // [M-1][RG]
    int32_t *filled;         // [M-1][RG]
    int32_t *cell_to;        // [M-1][K]
    int32_t *out;            // [M-1][N] candidate layouts
    int32_t *ok;             // [M-1]
};

// (a before b) in RandomizedBestFit order: decreasing occupancy, then
// cardinality, then index.
__device__ inline bool fit_before(int64_t Ta, int32_t na, int32_t ca, int64_t Tb, int32_t nb, int32_t cb) {
    if (Ta != Tb) return Ta > Tb;
    if (na != nb) return na < nb;
    return ca < cb;
}
// (a before b) in EDPAwarePair insertion order.
__device__ inline bool pair_before(int64_t ia, int64_t pa, int32_t ha, int64_t ib, int64_t pb, int32_t hb) {
    if (ia != ib) return ia < ib;
    if (pa != pb) return pa < pb;
    return ha < hb;
}

__global__ void __launch_bounds__(64) k_pack_trials(TrialArgs a) {
    __shared__ int64_t sT[kMaxCells];
    __shared__ int32_t sN[kMaxCells];
    const int lane = lane_id();
    const int b = blockIdx.x;  // 0: x_paired; >= 1: trial b
    const int32_t N = a.N, K = a.K, RG = a.RG, LP = a.LP, L = a.L, P = a.P, G = a.G, D = a.D;
    int32_t *cellk = a.cellk + (int64_t)b * N;
    int32_t *Qc = a.Qc + (int64_t)b * K * LP;
    int64_t *peak = a.peak + (int64_t)b * K;
    int32_t *order = a.order + (int64_t)b * K;
    int32_t *Wt = a.Wt + (int64_t)b * RG * LP;
    int64_t *base = a.base + (int64_t)b * RG, *after = a.after + (int64_t)b * RG, *pkv = a.pkv + (int64_t)b * RG;
    int32_t *filled = a.filled + (int64_t)b * RG;
    int32_t *cell_to = a.cell_to + (int64_t)b * K;
    int32_t *out = a.out + (int64_t)b * N;
    const int32_t w = b == 0 ? 1 : a.w;
    const uint64_t *wd = b == 0 ? nullptr : a.words + (int64_t)(b - 1) * (2 * (int64_t)N + K);

    if (b == 0) {
        for (int32_t i = lane; i < N; i += kWave) cellk[i] = a.x_length[i];
    } else {
        // WindowShuffle: the window holds the first min(w, remaining) items of
        // the remaining (-t, i) order; item h is window[bounded(word, |window|)].
        int32_t win = lane < w && lane < N ? a.sigma[lane] : -1;
        int32_t next = w < N ? w : N;
        int32_t wsize = next;
        for (int32_t c = lane; c < K; c += kWave) {
            sT[c] = 0;
            sN[c] = 0;
        }
        __syncthreads();
        int32_t good = 1;
        for (int32_t h = 0; h < N; ++h) {
            const int32_t pos = (int32_t)bounded(wd[h], (uint64_t)wsize);
            const int32_t item = __shfl(win, pos, kWave);
            // remove position pos, append the next sigma item
            const int32_t up = __shfl(win, lane + 1 < kWave ? lane + 1 : lane, kWave);
            if (lane >= pos && lane < wsize - 1) win = up;
            if (next < N) {
                if (lane == wsize - 1) win = a.sigma[next];
                ++next;
            } else {
                if (lane == wsize - 1) win = -1;
                --wsize;
            }
            const int64_t ti = a.t[item];
            int32_t c;
            if (h < K) {
                c = h;
            } else {
                // RandomizedBestFit: rank the feasible cells and take the
                // rho-th of the leading min(w, |F|).
                // (uniform trip count: every lane takes part in each ballot)
                int32_t nf = 0;
                int64_t bT = -1; int32_t bn = 0, bc = -1;
                for (int32_t cb = 0; cb < K; cb += kWave) {
                    const int32_t cc = cb + lane;
                    const bool f = cc < K && sT[cc] + ti <= a.C;
                    if (f && (bc < 0 || fit_before(sT[cc], sN[cc], cc, bT, bn, bc))) {
                        bT = sT[cc]; bn = sN[cc]; bc = cc;
                    }
                    nf += __popcll(__ballot(f));
                }
                if (nf == 0) {
                    good = 0;
                    break;
                }
                const int32_t wp = w < nf ? w : nf;
                const int32_t rho = (int32_t)bounded(wd[N + h], (uint64_t)wp);
                int64_t pT = 0; int32_t pn = 0, pc = -1;
                for (int32_t pass = 0; pass <= rho; ++pass) {
                    if (pass > 0) {
                        // first feasible cell strictly after the previous pick
                        bT = -1; bn = 0; bc = -1;
                        for (int32_t cc = lane; cc < K; cc += kWave) {
                            const bool f = sT[cc] + ti <= a.C && fit_before(pT, pn, pc, sT[cc], sN[cc], cc);
                            if (f && (bc < 0 || fit_before(sT[cc], sN[cc], cc, bT, bn, bc))) {
                                bT = sT[cc]; bn = sN[cc]; bc = cc;
                            }
                        }
                    }
#pragma unroll
                    for (int d = 32; d >= 1; d >>= 1) {
                        const int64_t oT = __shfl_xor(bT, d, kWave);
                        const int32_t on = __shfl_xor(bn, d, kWave), oc = __shfl_xor(bc, d, kWave);
                        if (oc >= 0 && (bc < 0 || fit_before(oT, on, oc, bT, bn, bc))) {
                            bT = oT; bn = on; bc = oc;
                        }
                    }
                    pT = bT; pn = bn; pc = bc;
                }
                c = pc;
            }
            if (lane == 0) {
                sT[c] += ti;
                sN[c] += 1;
                cellk[item] = c;
            }
            __syncthreads();
        }
        if (!good) {
            if (lane == 0) a.ok[b] = 0;
            return;
        }
    }
    __syncthreads();
    // EDPAwarePair.  Q_k = sum of member rows; peak_k = sum_l max_p Q_k.
    for (int64_t x = lane; x < (int64_t)K * LP; x += kWave) Qc[x] = 0;
    __syncthreads();
    for (int32_t i = 0; i < N; ++i) {
        const int32_t k = cellk[i];
        const int32_t *qi = a.q + (int64_t)i * LP;
        for (int32_t e = lane; e < LP; e += kWave) Qc[(int64_t)k * LP + e] += qi[e];
    }
    __syncthreads();
    for (int32_t k = lane; k < K; k += kWave) {
        int64_t pk = 0;
        for (int l = 0; l < L; ++l) {
            int32_t mx = Qc[(int64_t)k * LP + l * P];
            for (int p = 1; p < P; ++p) mx = max(mx, Qc[(int64_t)k * LP + l * P + p]);
            pk += mx;
        }
        peak[k] = pk;
    }
    __syncthreads();
    for (int32_t k = lane; k < K; k += kWave) {
        const int64_t v = peak[k];
        int32_t rank = 0;
        for (int32_t f = 0; f < K; ++f) {
            const int64_t u = peak[f];
            rank += (u > v) || (u == v && f < k);
        }
        order[rank] = k;
    }
    for (int64_t x = lane; x < (int64_t)RG * LP; x += kWave) Wt[x] = 0;
    for (int32_t h = lane; h < RG; h += kWave) {
        base[h] = 0;
        filled[h] = 0;
    }
    __syncthreads();
    for (int32_t pos = 0; pos < K; ++pos) {
        const int32_t k = order[pos];
        const int32_t *Qk = Qc + (int64_t)k * LP;
        int32_t cnt = 0;
        for (int32_t hb = 0; hb < RG; hb += kWave) {
            const int32_t h = hb + lane;
            const bool cand = h < RG && filled[h] < a.count[h % G];
            int64_t af = 0, pk = 0;
            if (cand) {
                const int32_t *Wh = Wt + (int64_t)h * LP;
                for (int l = 0; l < L; ++l) {
                    int32_t mx = Wh[l * P] + Qk[l * P];
                    for (int p = 1; p < P; ++p) mx = max(mx, Wh[l * P + p] + Qk[l * P + p]);
                    af += mx;
                    pk = mx > pk ? mx : pk;
                }
            }
            if (h < RG) {
                after[h] = af;
                pkv[h] = pk;
            }
            cnt += __popcll(__ballot(cand));
        }
        __syncthreads();
        const int32_t wp = w < cnt ? w : cnt;
        int32_t rho = 0;
        if (wp > 1) {
            const uint64_t total = (((uint64_t)1) << wp) - 1;
            const uint64_t pick = bounded(wd[2 * (int64_t)N + pos], total);
            uint64_t pref = 0;
            for (rho = 0; rho < wp; ++rho) {
                pref += ((uint64_t)1) << (wp - 1 - rho);
                if (pref > pick) break;
            }
        }
        int64_t pI = 0, pP = 0;
        int32_t pH = -1;
        for (int32_t pass = 0; pass <= rho; ++pass) {
            int64_t bI = 0, bP = 0;
            int32_t bH = -1;
            for (int32_t h = lane; h < RG; h += kWave) {
                if (filled[h] >= a.count[h % G]) continue;
                const int64_t ih = after[h] - base[h], ph = pkv[h];
                if (pass > 0 && !pair_before(pI, pP, pH, ih, ph, h)) continue;
                if (bH < 0 || pair_before(ih, ph, h, bI, bP, bH)) {
                    bI = ih; bP = ph; bH = h;
                }
            }
#pragma unroll
            for (int d = 32; d >= 1; d >>= 1) {
                const int64_t oI = __shfl_xor(bI, d, kWave), oP = __shfl_xor(bP, d, kWave);
                const int32_t oH = __shfl_xor(bH, d, kWave);
                if (oH >= 0 && (bH < 0 || pair_before(oI, oP, oH, bI, bP, bH))) {
                    bI = oI; bP = oP; bH = oH;
                }
            }
            pI = bI; pP = bP; pH = bH;
        }
        const int32_t h = pH;
        const int32_t r = h / G, g = h % G;
        const int32_t d = a.slots[g * D + filled[h]];
        int32_t *Wh = Wt + (int64_t)h * LP;
        for (int32_t e = lane; e < LP; e += kWave) Wh[e] += Qk[e];
        __syncthreads();
        if (lane == 0) {
            base[h] = after[h];
            filled[h] += 1;
            cell_to[k] = r * D + d;
        }
        __syncthreads();
    }
    for (int32_t i = lane; i < N; i += kWave) out[i] = cell_to[cellk[i]];
    if (lane == 0) a.ok[b] = 1;
}

// ---------------------------------------------------------------------------
// Seed trials in three launches for the common shapes (C < 2^31, N and K
// below 2^16, the pairing's tables other than W within LDS); the
// single-kernel path above covers the rest.  Same draws, same decisions.
//
//  k_pack_fit      one wave per candidate: WindowShuffle and
//                  RandomizedBestFit with the draws, window items and their
//                  lengths prefetched 64 steps ahead into lane registers; the
//                  ranked pick compares 64-bit keys (load, then fewer
//                  members, then lower index) with DPP maxima.  Ends with the
//                  member list of every cell.  k_pack_fit_reg keeps the keys
//                  in registers up to 2048 cells, k_pack_fit in LDS above.
//  k_pack_cellsum  one workgroup per (candidate, cell): Q_k = sum of the
//                  member rows and peak_k = sum_l max_p Q_k.
//  k_pack_pair     one workgroup per candidate: EDPAwarePair with the W table
//                  in LDS when it fits (else in the trial's slice of HBM),
//                  threads over 4 consecutive entries of W + Q_k and a DPP
//                  maximum over each layer's ranks, and the next cell's Q
//                  row prefetched during each step.

struct PackFast {
    int32_t *mstart;  // [M-1][K+1] member list offsets
    int32_t *mlist;   // [M-1][N] members, grouped by cell
};

// RandomizedBestFit key of a cell: a larger key comes first.
__device__ inline uint64_t fit_key(int64_t T, int32_t n, int32_t c) {
    return ((uint64_t)T << 32) | ((uint64_t)(0xFFFF - n) << 16) | (uint64_t)(0xFFFF - c);
}

__global__ void __launch_bounds__(64) k_pack_fit(TrialArgs a, PackFast pf) {
    extern __shared__ int64_t sfit[];
    const int lane = lane_id();
    const int b = blockIdx.x;
    const int32_t N = a.N, K = a.K;
    int64_t *sT = sfit;
    int32_t *sN = reinterpret_cast<int32_t *>(sT + K);
    int32_t *cur = sN + K;
    int32_t *cellk = a.cellk + (int64_t)b * N;
    for (int32_t c = lane; c < K; c += kWave) {
        sT[c] = 0;
        sN[c] = 0;
    }
    __syncthreads();
    int32_t good = 1;
    if (b == 0) {
        for (int32_t i = lane; i < N; i += kWave) {
            const int32_t c = a.x_length[i];
            cellk[i] = c;
            atomicAdd(&sN[c], 1);
        }
    } else {
        const int32_t w = a.w;
        const uint64_t *wd = a.words + (int64_t)(b - 1) * (2 * (int64_t)N + K);
        // window: lane x < wsize holds item x and its length
        int32_t win = -1, wint = 0;
        if (lane < w && lane < N) {
            win = a.sigma[lane];
            wint = a.t[win];
        }
        int32_t next = w < N ? w : N, wsize = next;
        // prefetched sigma items entering the window, with their lengths
        int32_t sbase = next;
        int32_t sreg = sbase + lane < N ? a.sigma[sbase + lane] : 0;
        int32_t streg = sbase + lane < N ? a.t[sreg] : 0;
        // prefetched draws: shuffle word h and best-fit word h
        int32_t hbase = 0;
        uint64_t wr1 = lane < N ? wd[lane] : 0, wr2 = lane < N ? wd[N + lane] : 0;
        for (int32_t h = 0; h < N; ++h) {
            if (h - hbase == kWave) {
                hbase += kWave;
                wr1 = hbase + lane < N ? wd[hbase + lane] : 0;
                wr2 = hbase + lane < N ? wd[N + hbase + lane] : 0;
            }
            const int32_t pos = (int32_t)bounded(readlane64(wr1, h - hbase), (uint64_t)wsize);
            const int32_t item = __builtin_amdgcn_readlane(win, pos);
            const int64_t ti = __builtin_amdgcn_readlane(wint, pos);
            // remove position pos, append the next sigma item
            int32_t up, upt;
            if (w <= 16) {  // row_shl:1 -- lane i reads lane i + 1 of its 16-lane row
                up = __builtin_amdgcn_update_dpp(win, win, 0x101, 0xF, 0xF, false);
                upt = __builtin_amdgcn_update_dpp(wint, wint, 0x101, 0xF, 0xF, false);
            } else {
                up = __shfl_down(win, 1, kWave);
                upt = __shfl_down(wint, 1, kWave);
            }
            if (lane >= pos && lane < wsize - 1) {
                win = up;
                wint = upt;
            }
            if (next < N) {
                if (next - sbase == kWave) {
                    sbase += kWave;
                    sreg = sbase + lane < N ? a.sigma[sbase + lane] : 0;
                    streg = sbase + lane < N ? a.t[sreg] : 0;
                }
                const int32_t ni = __builtin_amdgcn_readlane(sreg, next - sbase);
                const int32_t nt = __builtin_amdgcn_readlane(streg, next - sbase);
                if (lane == wsize - 1) {
                    win = ni;
                    wint = nt;
                }
                ++next;
            } else {
                if (lane == wsize - 1) {
                    win = -1;
                    wint = 0;
                }
                --wsize;
            }
            int32_t c;
            if (h < K) {
                c = h;
            } else {
                uint64_t best = 0;
                int32_t nf = 0;
                for (int32_t cb = 0; cb < K; cb += kWave) {
                    const int32_t cc = cb + lane;
                    const bool f = cc < K && sT[cc] + ti <= a.C;
                    nf += __popcll(__ballot(f));
                    if (f) {
                        const uint64_t k = fit_key(sT[cc], sN[cc], cc);
                        best = k > best ? k : best;
                    }
                }
                if (nf == 0) {
                    good = 0;
                    break;
                }
                best = wave_max_u64(best);
                const int32_t wp = w < nf ? w : nf;
                const int32_t rho = (int32_t)bounded(readlane64(wr2, h - hbase), (uint64_t)wp);
                for (int32_t pass = 1; pass <= rho; ++pass) {
                    const uint64_t prev = best;
                    best = 0;
                    for (int32_t cb = 0; cb < K; cb += kWave) {
                        const int32_t cc = cb + lane;
                        if (cc < K && sT[cc] + ti <= a.C) {
                            const uint64_t k = fit_key(sT[cc], sN[cc], cc);
                            if (k < prev && k > best) best = k;
                        }
                    }
                    best = wave_max_u64(best);
                }
                c = 0xFFFF - (int32_t)(best & 0xFFFF);
            }
            if (lane == 0) {
                sT[c] += ti;
                sN[c] += 1;
                cellk[item] = c;
            }
            __syncthreads();
        }
    }
    if (lane == 0) a.ok[b] = good;
    if (!good) return;
    __syncthreads();
    // member lists: offsets by an exclusive scan of the counts, then a scatter
    int32_t *ms = pf.mstart + (int64_t)b * (K + 1);
    int32_t *ml = pf.mlist + (int64_t)b * N;
    int64_t carry = 0;
    for (int32_t cb = 0; cb < K; cb += kWave) {
        const int32_t cc = cb + lane;
        const int64_t v = cc < K ? sN[cc] : 0;
        const int64_t incl = wave_incl_scan(v);
        if (cc < K) {
            ms[cc] = (int32_t)(carry + incl - v);
            cur[cc] = (int32_t)(carry + incl - v);
        }
        carry += (int64_t)readlane64((uint64_t)incl, kWave - 1);
    }
    if (lane == 0) ms[K] = N;
    __syncthreads();
    for (int32_t i = lane; i < N; i += kWave) {
        const int32_t c = cellk[i];
        ml[atomicAdd(&cur[c], 1)] = i;
    }
}

// k_pack_fit for K <= 64 NCH cells: lane x holds the keys of cells x,
// x + 64, ... in registers, so the ranked passes need no LDS traffic and a
// placement updates one lane.  A key carries the load in its high 32 bits
// (C < 2^31) and 0xFFFF - members below, so "the item fits" is one compare,
// key < (C - t + 1) << 32, and a placement adds (t << 32) - (1 << 16).  The
// draws, the window's next items and their lengths are loaded one block of
// 64 steps ahead, and each step's (item, cell) stays in the register of lane
// (step mod 64) until its block ends, so no step waits on memory.
template <int NCH>
__global__ void __launch_bounds__(64) k_pack_fit_reg(TrialArgs a, PackFast pf) {
    extern __shared__ int32_t sfitr[];  // [K] counts, then [K] cursors
    const int lane = lane_id();
    const int b = blockIdx.x;
    const int32_t N = a.N, K = a.K;
    int32_t *cnt_s = sfitr, *cur = sfitr + K;
    int32_t *cellk = a.cellk + (int64_t)b * N;
    uint64_t kr[NCH];
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
        const int32_t c = u * kWave + lane;
        kr[u] = c < K ? fit_key(0, 0, c) : ~(uint64_t)0;  // a missing cell never fits
    }
    int32_t good = 1;
    if (b == 0) {
        for (int32_t c = lane; c < K; c += kWave) cnt_s[c] = 0;
        __syncthreads();
        for (int32_t i = lane; i < N; i += kWave) {
            const int32_t c = a.x_length[i];
            cellk[i] = c;
            atomicAdd(&cnt_s[c], 1);
        }
    } else {
        const int32_t w = a.w;
        const uint64_t *wd = a.words + (int64_t)(b - 1) * (2 * (int64_t)N + K);
        int32_t win = -1, wint = 0;
        if (lane < w && lane < N) {
            win = a.sigma[lane];
            wint = a.t[win];
        }
        int32_t next = w < N ? w : N, wsize = next;
        // items entering the window: this block (s0, t0), the next (s1, t1)
        // and the items of the one after (s2), whose lengths are loaded when
        // it becomes the next
        int32_t sbase = next;
        const int32_t i0 = sbase + lane, i1 = i0 + kWave, i2 = i1 + kWave;
        int32_t s0 = i0 < N ? a.sigma[i0] : 0, s1 = i1 < N ? a.sigma[i1] : 0;
        int32_t s2 = i2 < N ? a.sigma[i2] : 0;
        int32_t t0 = i0 < N ? a.t[s0] : 0, t1 = i1 < N ? a.t[s1] : 0;
        // draws: shuffle word h and best-fit word h, this block and the next
        int32_t hbase = 0;
        uint64_t wr1 = lane < N ? wd[lane] : 0, wr2 = lane < N ? wd[N + lane] : 0;
        uint64_t nw1 = kWave + lane < N ? wd[kWave + lane] : 0;
        uint64_t nw2 = kWave + lane < N ? wd[N + kWave + lane] : 0;
        // Step hb + lane's window position (the window holds min(w, N - h)
        // items at step h) and its rank when w or more cells fit, drawn when
        // the block becomes current.
        auto draws = [&](int32_t hb, int32_t &pos_l, int32_t &rho_l) {
            const int32_t hh = hb + lane, ws = w < N - hh ? w : N - hh;
            pos_l = hh < N ? (int32_t)bounded(wr1, (uint64_t)ws) : 0;
            rho_l = (int32_t)bounded(wr2, (uint64_t)w);
        };
        int32_t pos_l, rho_l;
        draws(0, pos_l, rho_l);
        int32_t p_item = -1, p_cell = 0;  // step hbase + lane's placement
        for (int32_t h = 0; h < N; ++h) {
            if (h - hbase == kWave) {
                if (p_item >= 0) cellk[p_item] = p_cell;
                p_item = -1;
                hbase += kWave;
                wr1 = nw1;
                wr2 = nw2;
                draws(hbase, pos_l, rho_l);
                const int32_t hn = hbase + kWave + lane;
                nw1 = hn < N ? wd[hn] : 0;
                nw2 = hn < N ? wd[N + hn] : 0;
            }
            const int32_t pos = __builtin_amdgcn_readlane(pos_l, h - hbase);
            const int32_t item = __builtin_amdgcn_readlane(win, pos);
            const int32_t ti = __builtin_amdgcn_readlane(wint, pos);
            int32_t up, upt;
            if (w <= 16) {  // row_shl:1 -- lane i reads lane i + 1 of its 16-lane row
                up = __builtin_amdgcn_update_dpp(win, win, 0x101, 0xF, 0xF, false);
                upt = __builtin_amdgcn_update_dpp(wint, wint, 0x101, 0xF, 0xF, false);
            } else {
                up = __shfl_down(win, 1, kWave);
                upt = __shfl_down(wint, 1, kWave);
            }
            if (lane >= pos && lane < wsize - 1) {
                win = up;
                wint = upt;
            }
            if (next < N) {
                if (next - sbase == kWave) {
                    sbase += kWave;
                    s0 = s1;
                    t0 = t1;
                    s1 = s2;
                    const int32_t j1 = sbase + kWave + lane, j2 = j1 + kWave;
                    t1 = j1 < N ? a.t[s1] : 0;
                    s2 = j2 < N ? a.sigma[j2] : 0;
                }
                const int32_t ni = __builtin_amdgcn_readlane(s0, next - sbase);
                const int32_t nt = __builtin_amdgcn_readlane(t0, next - sbase);
                if (lane == wsize - 1) {
                    win = ni;
                    wint = nt;
                }
                ++next;
            } else {
                if (lane == wsize - 1) {
                    win = -1;
                    wint = 0;
                }
                --wsize;
            }
            int32_t c;
            if (h < K) {
                c = h;
            } else {
                const uint64_t lim = ti <= a.C ? (uint64_t)(a.C - ti + 1) << 32 : 0;
                uint64_t best = 0;
                int32_t nf = 0;
#pragma unroll
                for (int u = 0; u < NCH; ++u) {
                    const bool f = kr[u] < lim;
                    nf += __popcll(__ballot(f));
                    if (f && kr[u] > best) best = kr[u];
                }
                if (nf == 0) {
                    good = 0;
                    break;
                }
                best = wave_max_u64(best);
                const int32_t rho = nf >= w ? __builtin_amdgcn_readlane(rho_l, h - hbase)
                                            : (int32_t)bounded(readlane64(wr2, h - hbase), (uint64_t)nf);
                // a key below a fitting key fits too
                for (int32_t pass = 1; pass <= rho; ++pass) {
                    const uint64_t prev = best;
                    best = 0;
#pragma unroll
                    for (int u = 0; u < NCH; ++u)
                        if (kr[u] < prev && kr[u] > best) best = kr[u];
                    best = wave_max_u64(best);
                }
                c = 0xFFFF - (int32_t)(best & 0xFFFF);
            }
            // c is uniform: only its chunk's owner lane changes (a select per
            // chunk, so every register index stays static)
            const int32_t cu = c >> 6;
            const bool own = (c & (kWave - 1)) == lane;
            const uint64_t add = own ? ((uint64_t)(uint32_t)ti << 32) - ((uint64_t)1 << 16) : 0;
#pragma unroll
            for (int u = 0; u < NCH; ++u) kr[u] += u == cu ? add : 0;
            if (lane == h - hbase) {
                p_item = item;
                p_cell = c;
            }
        }
        if (p_item >= 0) cellk[p_item] = p_cell;
#pragma unroll
        for (int u = 0; u < NCH; ++u)
            if (u * kWave + lane < K) cnt_s[u * kWave + lane] = 0xFFFF - (int32_t)((kr[u] >> 16) & 0xFFFF);
    }
    if (lane == 0) a.ok[b] = good;
    if (!good) return;
    __syncthreads();
    int32_t *ms = pf.mstart + (int64_t)b * (K + 1);
    int32_t *ml = pf.mlist + (int64_t)b * N;
    int64_t carry = 0;
    for (int32_t cb = 0; cb < K; cb += kWave) {
        const int32_t cc = cb + lane;
        const int64_t v = cc < K ? cnt_s[cc] : 0;
        const int64_t incl = wave_incl_scan(v);
        if (cc < K) {
            ms[cc] = (int32_t)(carry + incl - v);
            cur[cc] = (int32_t)(carry + incl - v);
        }
        carry += (int64_t)readlane64((uint64_t)incl, kWave - 1);
    }
    if (lane == 0) ms[K] = N;
    __syncthreads();
    for (int32_t i = lane; i < N; i += kWave) {
        const int32_t c = cellk[i];
        ml[atomicAdd(&cur[c], 1)] = i;
    }
}

// Q_k and peak_k of cell k = blockIdx.x of candidate b = blockIdx.y.
__global__ void __launch_bounds__(128) k_pack_cellsum(TrialArgs a, PackFast pf) {
    extern __shared__ int32_t sq[];
    __shared__ int64_t spart[4];
    const int b = blockIdx.y, k = blockIdx.x, tid = threadIdx.x, nt = blockDim.x;
    if (!a.ok[b]) return;  // uniform: a failed trial has no layout
    const int32_t K = a.K, LP = a.LP, L = a.L, P = a.P;
    const int32_t *ms = pf.mstart + (int64_t)b * (K + 1);
    const int32_t *ml = pf.mlist + (int64_t)b * a.N;
    const int32_t lo = ms[k], hi = ms[k + 1];
    int32_t *Qk = a.Qc + ((int64_t)b * K + k) * LP;
    for (int32_t e = tid; e < LP; e += nt) {
        int32_t acc = 0;
        for (int32_t x = lo; x < hi; ++x) acc += a.q[(int64_t)ml[x] * LP + e];
        Qk[e] = acc;
        sq[e] = acc;
    }
    __syncthreads();
    int64_t part = 0;
    for (int32_t l = tid; l < L; l += nt) {
        int32_t mx = sq[l * P];
        for (int32_t p = 1; p < P; ++p) mx = max(mx, sq[l * P + p]);
        part += mx;
    }
    part = wave_sum(part);
    if (lane_id() == 0) spart[wave_id()] = part;
    __syncthreads();
    if (tid == 0) {
        int64_t tot = 0;
        for (int w = 0; w < nt / kWave; ++w) tot += spart[w];
        a.peak[(int64_t)b * K + k] = tot;
    }
}

// EDPAwarePair of candidate b (block per candidate).
// WG: the trial's row-shard loads W stay in its slice of a.Wt in HBM (when
// they do not fit LDS next to the rest); every W access is a coalesced
// 16-byte read or an update of one row by the whole workgroup.
template <bool WG>
__global__ void __launch_bounds__(1024) k_pack_pair(TrialArgs a, PackFast pf) {
    extern __shared__ __align__(16) char spair[];
    __shared__ int32_t s_h;
    const int b = blockIdx.x, tid = threadIdx.x, nt = blockDim.x, lane = lane_id(), wv = wave_id();
    if (!a.ok[b]) return;  // uniform
    const int32_t N = a.N, K = a.K, RG = a.RG, LP = a.LP, L = a.L, P = a.P, G = a.G, D = a.D;
    const int32_t w = b == 0 ? 1 : a.w;
    const uint64_t *wd = b == 0 ? nullptr : a.words + (int64_t)(b - 1) * (2 * (int64_t)N + K);
    int64_t *after = reinterpret_cast<int64_t *>(spair);            // [RG]
    int64_t *pkv = after + RG, *base = pkv + RG;                    // [RG], [RG]
    int64_t *speak = base + RG;                                     // [K]
    int32_t *lds_next = reinterpret_cast<int32_t *>(speak + K + ((3 * RG + K) & 1));  // 16-byte aligned
    int32_t *Wl = WG ? a.Wt + (int64_t)b * RG * LP : lds_next;      // [RG][LP]
    int32_t *qb = WG ? lds_next : Wl + (int64_t)RG * LP;            // [2][LP]
    int32_t *mxs = qb + 2 * LP;                                     // [RG][L]
    int32_t *filled = mxs + RG * L;                                 // [RG]
    int32_t *hcnt = filled + RG;                                    // [RG]
    int32_t *order = hcnt + RG;                                     // [K]
    int32_t *cell_to = order + K;                                   // [K]
    const int32_t *Qc = a.Qc + (int64_t)b * K * LP;
    for (int32_t k = tid; k < K; k += nt) speak[k] = a.peak[(int64_t)b * K + k];
    for (int64_t x = tid; x < (int64_t)RG * LP; x += nt) Wl[x] = 0;
    for (int32_t h = tid; h < RG; h += nt) {
        base[h] = 0;
        filled[h] = 0;
        hcnt[h] = a.count[h % G];
    }
    __syncthreads();
    // order: cells by decreasing peak, then index
    for (int32_t k = tid; k < K; k += nt) {
        const int64_t v = speak[k];
        int32_t rank = 0;
        for (int32_t f = 0; f < K; ++f) {
            const int64_t u = speak[f];
            rank += (u > v) || (u == v && f < k);
        }
        order[rank] = k;
    }
    __syncthreads();
    for (int32_t e = tid; e < LP; e += nt) qb[e] = Qc[(int64_t)order[0] * LP + e];
    __syncthreads();
    constexpr int kPre = 16;  // Q entries per thread held for the next step (LP <= 16 * 1024)
    uint64_t wpair = 0;       // wave 0: pairing draws of steps pbase .. pbase + 63, one per lane
    int32_t pbase = -kWave;
    for (int32_t pos = 0; pos < K; ++pos) {
        if (wv == 0 && wd && pos - pbase == kWave) {
            pbase = pos;
            wpair = pos + lane < K ? wd[2 * (int64_t)N + pos + lane] : 0;
        }
        const int32_t k = order[pos];
        const int32_t *qk = qb + (pos & 1) * LP;
        // next cell's Q row into registers while this step runs
        int32_t nq[kPre];
        const bool more = pos + 1 < K;
        const int64_t nrow = more ? (int64_t)order[pos + 1] * LP : 0;
#pragma unroll
        for (int u = 0; u < kPre; ++u) {
            const int32_t e = tid + u * nt;
            nq[u] = more && e < LP ? Qc[nrow + e] : 0;
        }
        // per (row-shard, layer): max over ranks of W + Q_k; a thread holds 4
        // consecutive entries, a layer's ranks span P / 4 adjacent threads.
        // Every thread runs the same number of iterations, so the DPP maximum
        // always sees its whole group.
        {
            const int32_t c4 = LP >> 2, g4 = P >> 2;
            const int32_t iters = (RG * c4 + nt - 1) / nt;
            int32_t y = tid, h = 0;
            while (y >= c4) {
                y -= c4;
                ++h;
            }
            for (int32_t it = 0; it < iters; ++it) {
                const bool cand = h < RG && filled[h] < hcnt[h];
                int32_t mx = INT32_MIN;
                if (cand) {
                    const int4 wv4 = reinterpret_cast<const int4 *>(Wl + (int64_t)h * LP)[y];
                    const int4 qv4 = reinterpret_cast<const int4 *>(qk)[y];
                    mx = max(max(wv4.x + qv4.x, wv4.y + qv4.y), max(wv4.z + qv4.z, wv4.w + qv4.w));
                }
                mx = seg_max32(mx, g4);
                if (cand && (y & (g4 - 1)) == 0) mxs[h * L + y / g4] = mx;
                y += nt;
                while (y >= c4) {
                    y -= c4;
                    ++h;
                }
            }
        }
        __syncthreads();
        for (int32_t h = tid; h < RG; h += nt) {
            int64_t af = 0, pk = 0;
            if (filled[h] < hcnt[h]) {
                if ((L & 3) == 0) {  // the row's maxima as 16-byte reads (mxs is 16-byte aligned)
                    const int4 *m4 = reinterpret_cast<const int4 *>(mxs + h * L);
                    for (int32_t l4 = 0; l4 < (L >> 2); ++l4) {
                        const int4 v = m4[l4];
                        af += (int64_t)v.x + v.y + v.z + v.w;
                        const int32_t m = max(max(v.x, v.y), max(v.z, v.w));
                        pk = m > pk ? m : pk;
                    }
                } else {
                    for (int32_t l = 0; l < L; ++l) {
                        const int32_t mx = mxs[h * L + l];
                        af += mx;
                        pk = mx > pk ? mx : pk;
                    }
                }
            }
            after[h] = af;
            pkv[h] = pk;
        }
        __syncthreads();
        if (wv == 0) {
            // candidates in EDPAwarePair order (increase, peak, index); the
            // rho-th of the leading min(w, |candidates|)
            int32_t cnt = 0;
            for (int32_t hb = 0; hb < RG; hb += kWave)
                cnt += __popcll(__ballot(hb + lane < RG && filled[hb + lane] < hcnt[hb + lane]));
            const int32_t wp = w < cnt ? w : cnt;
            int32_t rho = 0;
            if (wp > 1) {
                const uint64_t total = (((uint64_t)1) << wp) - 1;
                const uint64_t pick = bounded(readlane64(wpair, pos - pbase), total);
                uint64_t pref = 0;
                for (rho = 0; rho < wp; ++rho) {
                    pref += ((uint64_t)1) << (wp - 1 - rho);
                    if (pref > pick) break;
                }
            }
            int64_t p0 = LLONG_MIN, p1 = LLONG_MIN, p2 = LLONG_MIN;
            for (int32_t pass = 0; pass <= rho; ++pass) {
                int64_t k0 = LLONG_MAX, k1 = LLONG_MAX, k2 = LLONG_MAX, kj = LLONG_MAX;
                for (int32_t hb = 0; hb < RG; hb += kWave) {
                    const int32_t h = hb + lane;
                    if (h < RG && filled[h] < hcnt[h]) {
                        const int64_t v0 = after[h] - base[h], v1 = pkv[h], v2 = h;
                        if ((pass == 0 || lex_less(p0, p1, p2, v0, v1, v2)) && lex_less(v0, v1, v2, k0, k1, k2)) {
                            k0 = v0; k1 = v1; k2 = v2; kj = v2;
                        }
                    }
                }
                wave_lexmin(k0, k1, k2, kj);
                p0 = k0; p1 = k1; p2 = k2;
            }
            if (lane == 0) s_h = (int32_t)p2;
        }
        __syncthreads();
        const int32_t h = s_h;
        for (int32_t e = tid; e < LP; e += nt) Wl[(int64_t)h * LP + e] += qk[e];
        if (tid == 0) {
            const int32_t r = h / G, g = h - r * G;
            base[h] = after[h];
            cell_to[k] = r * D + a.slots[g * D + filled[h]];
            filled[h] += 1;
        }
        int32_t *qn = qb + ((pos + 1) & 1) * LP;
#pragma unroll
        for (int u = 0; u < kPre; ++u) {
            const int32_t e = tid + u * nt;
            if (more && e < LP) qn[e] = nq[u];
        }
        __syncthreads();
    }
    const int32_t *cellk = a.cellk + (int64_t)b * N;
    int32_t *out = a.out + (int64_t)b * N;
    for (int32_t i = tid; i < N; i += nt) out[i] = cell_to[cellk[i]];
}

// Canonical form of layouts[b] (b < n) into canon[b].
__global__ void __launch_bounds__(256) k_canonical(const int32_t *layouts, int32_t n, int32_t N, int32_t R,
                                                   int32_t D, int32_t G, const int32_t *slots,
                                                   const int32_t *count, const int32_t *slot_shard,
                                                   int32_t *cellmin_g, int32_t *newcell_g, int32_t *rowkey_g,
                                                   int32_t *canon) {
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    const int32_t B = R * D;
    const int32_t *lay = layouts + (int64_t)b * N;
    int32_t *cmin = cellmin_g + (int64_t)b * B;
    int32_t *newd = newcell_g + (int64_t)b * B;
    int32_t *rkey = rowkey_g + (int64_t)b * R;
    for (int32_t c = tid; c < B; c += blockDim.x) cmin[c] = INT32_MAX;
    __syncthreads();
    for (int32_t i = tid; i < N; i += blockDim.x) {
        const int32_t c = lay[i];
        if (c >= 0 && c < B) atomicMin(&cmin[c], i);
    }
    __syncthreads();
    // slot of each cell within its row-shard after ordering by smallest id
    for (int32_t c = tid; c < B; c += blockDim.x) {
        const int32_t r = c / D, d = c % D, g = slot_shard[d];
        const int32_t v = cmin[c];
        int32_t rank = 0;
        for (int32_t x = 0; x < count[g]; ++x) {
            const int32_t u = cmin[r * D + slots[g * D + x]];
            rank += u < v;
        }
        newd[c] = slots[g * D + rank];
    }
    __syncthreads();
    // row key: smallest id of the cell that lands in slot 0
    for (int32_t r = tid; r < R; r += blockDim.x) rkey[r] = INT32_MAX;
    __syncthreads();
    for (int32_t c = tid; c < B; c += blockDim.x)
        if (newd[c] == 0) rkey[c / D] = cmin[c];
    __syncthreads();
    for (int32_t c = tid; c < B; c += blockDim.x) {
        const int32_t r = c / D;
        const int32_t v = rkey[r];
        int32_t rank = 0;
        for (int32_t x = 0; x < R; ++x) rank += rkey[x] < v;
        newd[c] = rank * D + newd[c];
    }
    __syncthreads();
    for (int32_t i = tid; i < N; i += blockDim.x) {
        const int32_t c = lay[i];
        canon[(int64_t)b * N + i] = (c >= 0 && c < B) ? newd[c] : -1;
    }
}

// Selection and cyclic fill.  cand m: 0 x_length, 1 x_paired (kept when
// strictly better than x_length), m >= 2 trial m-1 (kept when it succeeded).
__global__ void __launch_bounds__(256) k_pack_select(const int32_t *canon, const int64_t *scores,
                                                     const int32_t *ok, const int32_t *status,
                                                     int32_t M, int32_t N,
                                                     int32_t *keep_order, int32_t *meta) {
    __shared__ int32_t valid[64], kept[64], order[64];
    __shared__ int32_t differ;
    const int tid = threadIdx.x;
    if (tid < M) {
        int32_t v = 1;
        if (tid == 1) {
            const int64_t *a = scores + 3, *x = scores;
            v = ok[0] && status[1] == 0 && lex_less(a[0], a[1], a[2], x[0], x[1], x[2]);
        } else if (tid >= 2) {
            v = ok[tid - 1] && status[tid] == 0;
        }
        valid[tid] = v;
        kept[tid] = 0;
    }
    __syncthreads();
    for (int m = 0; m < M; ++m) {
        if (!valid[m]) continue;
        bool dup = false;
        for (int u = 0; u < m && !dup; ++u) {
            if (!kept[u]) continue;
            if (tid == 0) differ = 0;
            __syncthreads();
            for (int32_t i = tid; i < N; i += blockDim.x)
                if (canon[(int64_t)m * N + i] != canon[(int64_t)u * N + i]) differ = 1;
            __syncthreads();
            dup = differ == 0;
            __syncthreads();
        }
        if (tid == 0) kept[m] = dup ? 0 : 1;
        __syncthreads();
    }
    if (tid == 0) {
        int32_t n = 0;
        for (int m = 0; m < M; ++m)
            if (kept[m]) order[n++] = m;
        // insertion sort by (score, discovery)
        for (int x = 1; x < n; ++x) {
            const int32_t v = order[x];
            int y = x - 1;
            while (y >= 0) {
                const int64_t *a = scores + 3 * (int64_t)order[y], *c = scores + 3 * (int64_t)v;
                if (lex_less(c[0], c[1], c[2], a[0], a[1], a[2])) {
                    order[y + 1] = order[y];
                    --y;
                } else {
                    break;
                }
            }
            order[y + 1] = v;
        }
        for (int x = 0; x < n; ++x) keep_order[x] = order[x];
        int32_t ntr = 0;
        for (int m = 2; m < M; ++m) ntr += ok[m - 1] && status[m] == 0;
        meta[0] = n;
        meta[1] = ntr;
    }
}

__global__ void k_pack_fill(const int32_t *canon, const int64_t *scores, const int32_t *keep_order,
                            const int32_t *meta, int32_t N, int32_t *population, int64_t *pop_scores) {
    const int m = blockIdx.x;
    const int32_t src = keep_order[m % meta[0]];
    for (int32_t i = threadIdx.x; i < N; i += blockDim.x)
        population[(int64_t)m * N + i] = canon[(int64_t)src * N + i];
    if (threadIdx.x < 3) pop_scores[(int64_t)m * 3 + threadIdx.x] = scores[(int64_t)src * 3 + threadIdx.x];
}

}  // namespace rp

namespace rp {
int rank_sort_desc(const int32_t *lengths, int32_t N, int32_t *sigma, hipStream_t stream) {
    hipLaunchKernelGGL(k_rank_sort, dim3((N + 255) / 256), dim3(256), 0, stream, lengths, N, sigma);
    return hipGetLastError() == hipSuccess ? ROUTEPACK_OK : ROUTEPACK_E_DEVICE;
}
}  // namespace rp

using namespace rp;

extern "C" int routepack_pack_rows(const routepack_problem *prob, const int32_t *lengths,
                                   const int32_t *q, uint64_t seed, int32_t n_trials,
                                   int32_t choice_width, int32_t pop_size, int32_t *r_star,
                                   int32_t *certified, int32_t *population, int64_t *scores,
                                   int32_t *info, hipStream_t stream) {
    Topology topo;
    RP_TRY(check_problem(prob, &topo));
    if (!lengths || (!q && prob->n_layers > 0) || !r_star || !certified || !population || !scores)
        return ROUTEPACK_E_INVALID;
    if (n_trials < 2 || n_trials > 64 || choice_width < 1 || choice_width > 62 || pop_size < 1)
        return ROUTEPACK_E_INVALID;
    const int32_t N = prob->n_samples, D = topo.D, G = topo.G;
    const int64_t C = prob->capacity;
    const int64_t LP = (int64_t)prob->n_layers * prob->n_ranks;
    if (LP > 4096) return ROUTEPACK_E_UNSUPPORTED;
    WindowStats ws;
    RP_TRY(window_stats(prob, lengths, q, &ws, stream));
    if (ws.q_negative) return ROUTEPACK_E_INVALID;
    if (ws.min_t < 1 || ws.max_t > C) return ROUTEPACK_E_INFEASIBLE;
    int64_t r_lb = prob->min_rows > 1 ? prob->min_rows : 1;
    const int64_t a1 = (ws.sum_t + C * D - 1) / (C * D);
    const int64_t a2 = (ws.n_big + D - 1) / D;
    r_lb = a1 > r_lb ? a1 : r_lb;
    r_lb = a2 > r_lb ? a2 : r_lb;
    const int64_t r_max = N / D;
    if (r_lb > r_max) return ROUTEPACK_E_INFEASIBLE;

    Scratch scr(stream);
    DeviceProblem dp;
    RP_TRY(upload_problem(prob, topo, scr, &dp, stream));
    int32_t *sigma = scr.get<int32_t>(N);
    int32_t *x_len = scr.get<int32_t>(N);
    int32_t *flag = scr.get<int32_t>(4);
    if (scr.failed()) return ROUTEPACK_E_DEVICE;
    hipLaunchKernelGGL(k_rank_sort, dim3((N + 255) / 256), dim3(256), 0, stream, lengths, N, sigma);
    int64_t R = -1;
    for (int64_t r = r_lb; r <= r_max; ++r) {
        if (r * D > kMaxCells) return ROUTEPACK_E_UNSUPPORTED;
        hipLaunchKernelGGL(k_ffd, dim3(1), dim3(64), 0, stream, lengths, sigma, N, C, (int32_t)(r * D),
                           x_len, flag);
        int32_t ok = 0;
        RP_HIP(hipMemcpyAsync(&ok, flag, sizeof(ok), hipMemcpyDeviceToHost, stream));
        RP_HIP(hipStreamSynchronize(stream));
        if (ok) {
            R = r;
            break;
        }
    }
    if (R < 0) return ROUTEPACK_E_HEURISTIC;
    RP_TRY(overflow_check(prob, R, ws, false));
    const int32_t K = (int32_t)(R * D), RG = (int32_t)(R * G), M = n_trials;
    const int32_t nb = M - 1;  // blocks: x_paired + trials 1..M-2
    uint64_t *words = scr.get<uint64_t>((size_t)(M - 2 > 0 ? M - 2 : 1) * (2 * (size_t)N + K));
    TrialArgs ta;
    memset(&ta, 0, sizeof(ta));
    ta.t = lengths; ta.q = q; ta.sigma = sigma; ta.x_length = x_len;
    ta.N = N; ta.L = prob->n_layers; ta.P = prob->n_ranks; ta.D = D; ta.G = G; ta.R = (int32_t)R;
    ta.K = K; ta.RG = RG; ta.LP = (int32_t)LP; ta.w = choice_width; ta.C = C;
    ta.slots = dp.slots; ta.count = dp.count; ta.words = words;
    ta.cellk = scr.get<int32_t>((size_t)nb * N);
    ta.Qc = scr.get<int32_t>((size_t)nb * K * (LP ? LP : 1));
    ta.peak = scr.get<int64_t>((size_t)nb * K);
    ta.order = scr.get<int32_t>((size_t)nb * K);
    ta.Wt = scr.get<int32_t>((size_t)nb * RG * (LP ? LP : 1));
    ta.base = scr.get<int64_t>((size_t)nb * RG);
    ta.after = scr.get<int64_t>((size_t)nb * RG);
    ta.pkv = scr.get<int64_t>((size_t)nb * RG);
    ta.filled = scr.get<int32_t>((size_t)nb * RG);
    ta.cell_to = scr.get<int32_t>((size_t)nb * K);
    // candidates: [0] x_length, [1..M-1] the blocks' layouts
    int32_t *cand = scr.get<int32_t>((size_t)M * N);
    int32_t *canon = scr.get<int32_t>((size_t)M * N);
    int64_t *cscore = scr.get<int64_t>((size_t)M * 3);
    int32_t *cstat = scr.get<int32_t>(M);
    int32_t *okv = scr.get<int32_t>(M);
    int32_t *cmin = scr.get<int32_t>((size_t)M * K);
    int32_t *newc = scr.get<int32_t>((size_t)M * K);
    int32_t *rkey = scr.get<int32_t>((size_t)M * R);
    int32_t *keep = scr.get<int32_t>(64);
    int32_t *meta = scr.get<int32_t>(2);
    if (scr.failed()) return ROUTEPACK_E_DEVICE;
    ta.out = cand + N;
    ta.ok = okv;
    if (M > 2)
        hipLaunchKernelGGL(k_seed_words, dim3(1024), dim3(256), 0, stream, seed, M, N, K, words);
    // every candidate slot starts as a valid layout (all samples in cell 0),
    // so a failed trial never leaves indices outside [0, R*D)
    hipLaunchKernelGGL(k_fill_i32, dim3(256), dim3(256), 0, stream, cand, (int64_t)M * N, 0);
    hipLaunchKernelGGL(k_fill_i32, dim3(1), dim3(64), 0, stream, okv, (int64_t)M, 0);
    RP_HIP(hipMemcpyAsync(cand, x_len, sizeof(int32_t) * N, hipMemcpyDeviceToDevice, stream));
    // Seed trials: three kernels for the common shapes, else one.
    // ROUTEPACK_PACK_KERNEL=single requests the single-kernel path.
    const char *pk_force = getenv("ROUTEPACK_PACK_KERNEL");
    // The pairing kernel keeps W in LDS when it fits (ROUTEPACK_PACK_W=hbm
    // keeps it in HBM regardless), else in HBM.
    const int64_t pair_rest = 8 * (3 * (int64_t)RG + K + 1) +
                              4 * (2 * LP + (int64_t)RG * prob->n_layers + 2 * (int64_t)RG + 2 * (int64_t)K);
    const char *pw_force = getenv("ROUTEPACK_PACK_W");
    const bool w_hbm = (pw_force && strcmp(pw_force, "hbm") == 0) || pair_rest + 4 * (int64_t)RG * LP > 150 * 1024;
    const int64_t pair_lds = pair_rest + (w_hbm ? 0 : 4 * (int64_t)RG * LP);
    const bool fast = !(pk_force && strcmp(pk_force, "single") == 0) && C < ((int64_t)1 << 31) && N < 65536 &&
                      prob->n_ranks >= 4 && LP > 0 && pair_lds <= 150 * 1024;
    if (fast) {
        PackFast pf;
        pf.mstart = scr.get<int32_t>((size_t)nb * (K + 1));
        pf.mlist = scr.get<int32_t>((size_t)nb * N);
        if (scr.failed()) return ROUTEPACK_E_DEVICE;
        const size_t fit_lds = (size_t)16 * K;
        RP_HIP(hipFuncSetAttribute((const void *)k_pack_fit, hipFuncAttributeMaxDynamicSharedMemorySize, (int)fit_lds));
        const void *pair_fn = w_hbm ? (const void *)k_pack_pair<true> : (const void *)k_pack_pair<false>;
        RP_HIP(hipFuncSetAttribute(pair_fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)pair_lds));
        if (K <= 8 * kWave) {
            hipLaunchKernelGGL(k_pack_fit_reg<8>, dim3(nb), dim3(64), (size_t)8 * K, stream, ta, pf);
        } else if (K <= 32 * kWave) {
            hipLaunchKernelGGL(k_pack_fit_reg<32>, dim3(nb), dim3(64), (size_t)8 * K, stream, ta, pf);
        } else {
            hipLaunchKernelGGL(k_pack_fit, dim3(nb), dim3(64), fit_lds, stream, ta, pf);
        }
        hipLaunchKernelGGL(k_pack_cellsum, dim3(K, nb), dim3(128), (size_t)4 * LP, stream, ta, pf);
        if (w_hbm) hipLaunchKernelGGL(k_pack_pair<true>, dim3(nb), dim3(1024), (size_t)pair_lds, stream, ta, pf);
        else hipLaunchKernelGGL(k_pack_pair<false>, dim3(nb), dim3(1024), (size_t)pair_lds, stream, ta, pf);
    } else {
        hipLaunchKernelGGL(k_pack_trials, dim3(nb), dim3(64), 0, stream, ta);
    }
    RP_HIP(hipGetLastError());
    // Score every candidate (failed trials leave garbage layouts: their
    // status is nonzero or they are ignored by the selection).
    RP_TRY(eval_layouts(prob, topo, dp, lengths, q, (int32_t)R, M, cand, cscore, cstat, nullptr,
                        nullptr, nullptr, stream));
    hipLaunchKernelGGL(k_canonical, dim3(M), dim3(256), 0, stream, cand, M, N, (int32_t)R, D, G,
                       dp.slots, dp.count, dp.slot_shard, cmin, newc, rkey, canon);
    hipLaunchKernelGGL(k_pack_select, dim3(1), dim3(256), 0, stream, canon, cscore, okv, cstat, M, N, keep,
                       meta);
    hipLaunchKernelGGL(k_pack_fill, dim3(pop_size), dim3(256), 0, stream, canon, cscore, keep, meta, N,
                       population, scores);
    RP_HIP(hipGetLastError());
    int32_t hmeta[2] = {0, 0};
    RP_HIP(hipMemcpyAsync(hmeta, meta, sizeof(hmeta), hipMemcpyDeviceToHost, stream));
    RP_HIP(hipStreamSynchronize(stream));
    *r_star = (int32_t)R;
    *certified = (R == r_lb) ? 1 : 0;
    if (info) {
        info[0] = (int32_t)r_lb;
        info[1] = hmeta[0];
        info[2] = hmeta[1];
    }
    return ROUTEPACK_OK;
}
