// Fixed-row population annealing (Alg. 3), one wave per population member,
// with the lanes laid out for the shape of one move rather than for a flat
// 64-entry stride.
//
// Layout of a move's work over the 64 lanes:
//  - W / q rows: lane (half, l) = (lane / 32, lane % 32) holds layer l (and
//    layer l + 32 when there are more than 32 layers) of row-shard a (half 0)
//    or b (half 1), all P ranks of each layer in registers, so the max over
//    ranks is in-lane and only the sum over layers crosses lanes (one 16-lane
//    DPP reduction per row-shard);
//  - cells: lane (half, x) with x < 16 holds the x-th cell of the row-shard,
//    so both attention maxima and both cell-cost prefixes come from one
//    16-lane DPP pass.
// Proposal screening is lane-parallel, as in the flat kernel, with a
// search structure that needs a fixed, small number of dependent LDS reads:
//  - the J roulette reads 8 pivots J_pre[8k+7] and then the 8 entries of one
//    block (two reads instead of a six-step binary search);
//  - the cell roulette reads the row-shard's cost prefix, stored
//    contiguously per row-shard, in one vector of reads.
// A relocation shifts the member pool through 32-bit words, four per lane
// (one 16-byte LDS access), instead of one 16-bit element per lane.
// The sequence of evaluated proposals, accept decisions and states is the
// sequential one (a rejected proposal leaves every screen valid, an accepted
// one triggers a re-screen of the rest of the batch).
#include <cstdlib>
#include <cstring>

#include "rp_anneal.h"

namespace rp {

namespace {

constexpr int64_t kInf = INT64_MAX;  // J prefix entries beyond the last row-shard

__device__ inline void wsync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Inclusive prefix sum over the first W lanes (W = 8 or 16) of each 16-lane
// row; W = 32: over each 32-lane half (rows 1 and 3 add the last lane of
// rows 0 and 2).
template <int W>
__device__ inline int64_t row_incl_scan64(int64_t v) {
    v += dpp64<kDppRowShr1>(v, 0);
    v += dpp64<kDppRowShr1 + 1>(v, 0);
    v += dpp64<kDppRowShr1 + 3>(v, 0);
    if (W > 8) v += dpp64<kDppRowShr1 + 7>(v, 0);
    if (W > 16) v += dpp64<kDppRowBcast15, 0xA>(v, 0);
    return v;
}

// Maximum over the first W lanes (W = 8 or 16) of each 16-lane row, held by
// those lanes; W = 32: over each 32-lane half, held by the lanes of rows 1
// and 3 (lanes 16 and 48 among them).
template <int W>
__device__ inline int64_t row_head_max64(int64_t v) {
    if (W > 16) {
        v = row_max64(v);
        const int64_t o = dpp64<kDppRowBcast15, 0xA>(v, v);
        return o > v ? o : v;
    }
    if (W > 8) return row_max64(v);
    int64_t o;
    o = dpp64<kDppXor1>(v, v); v = o > v ? o : v;
    o = dpp64<kDppXor2>(v, v); v = o > v ? o : v;
    o = dpp64<kDppHalfMirror>(v, v); v = o > v ? o : v;
    return v;
}

struct Lds {
    uint16_t *cell, *pool, *start;
    int32_t *gcell;  // the cell array in the member's slab instead (CG layout)
    int32_t *gpool;  // the pool in the member's slab instead (64 ranks)
    int32_t *T;
    int64_t *Q;
    // [RG][DV + 1] prefix of the cell costs of each row-shard, slot order;
    // kInf past its slots.  The odd row stride (in 8-byte words) spreads the
    // rows of a wave's random row reads over the LDS banks.
    int64_t *Cp;
    int64_t *Ctot;  // [RG] total cell cost of each row-shard
    int64_t *Jpre, *Vpre;  // [64 RV] prefixes of the source and target roulette weights (kInf past RG)
    int64_t *Jpiv, *Vpiv;  // [8 RV] their entries 8k+7
};

// Energy of a score (Eq. pa-energy); when the scale 2^F C is a power of two
// the three quotients are exact products with its reciprocal (identical
// results, no division).
__device__ inline double energy_k(const AnnealArgs &a, int64_t s0, int64_t s1, int64_t s2) {
    if (!a.scale_pow2) return energy(s0, s1, s2, a.scale);
    const double e0 = (double)s0 * a.inv_scale, e1 = (double)s1 * a.inv_scale, e2 = (double)s2 * a.inv_scale;
    const double x = e0 + 1e-6 * e1;
    return x + 1e-9 * e2;
}

// energy_k when the scale is known to be a power of two.
__device__ inline double energy_pow2(const AnnealArgs &a, int64_t s0, int64_t s1, int64_t s2) {
    const double e0 = (double)s0 * a.inv_scale, e1 = (double)s1 * a.inv_scale, e2 = (double)s2 * a.inv_scale;
    const double x = e0 + 1e-6 * e1;
    return x + 1e-9 * e2;
}

// floor(w m / 2^64) without a branch on the size of m (m varies by lane).
__device__ inline uint64_t bounded_lane(uint64_t w, uint64_t m) { return __umul64hi(w, m); }

// floor(x / d) for 0 <= x < 2^16 and 1 <= d < 2^16, with inv = ceil(2^32 / d)
// (exact: x d < 2^32); d == 1 is passed through.
__device__ inline int32_t div_small(int32_t x, int32_t d, uint32_t inv) {
    return d == 1 ? x : (int32_t)__umulhi((uint32_t)x, inv);
}

struct Tables {
    const int32_t *slots, *count, *shard, *soff, *t;
    const int32_t *hcnt;   // [RG] slots of each row-shard
    const int32_t *hcell;  // [RG][DV] cell of each slot of each row-shard
};

// Screen result of one proposal (per lane).
struct Screen {
    int32_t i, j, c1, c2, pos_i, pos_j, ti, tj;
    bool feas;
    // guided picks: source and target row-shards and the prefix entries
    // that bound each pick (J_pre[h1 - 1], J_pre[h1], V_pre[h4 - 1], V_pre[h4])
    int32_t h1, h4;
    int64_t jlo, jhi, vlo, vhi;
};

__device__ inline int32_t clamp0(int32_t v, int32_t hi) { return v < 0 ? 0 : (v > hi ? hi : v); }

// floor(w m / 2^64) for m < 2^32 (lane-varying m): hi(w) m plus the carry
// word floor(lo(w) m / 2^32), shifted down; both products are 32 x 32.
__device__ inline uint32_t bounded_small(uint64_t w, uint32_t m) {
    const uint64_t lo = (uint64_t)__umulhi((uint32_t)w, m);
    return (uint32_t)(((uint64_t)(uint32_t)(w >> 32) * m + lo) >> 32);
}

// A wave-uniform 64-bit value as scalar registers.
__device__ inline uint64_t uniform64(uint64_t v) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// floor(w m / 2^64) for a wave-uniform m (the branch on its size is scalar).
__device__ inline uint64_t bounded_uniform(uint64_t w, uint64_t m) {
    m = uniform64(m);
    if ((m >> 32) == 0) return bounded_small(w, (uint32_t)m);
    return __umul64hi(w, m);
}

// Ends a stage of independent LDS reads: every value listed is waited for
// here, so the reads of a stage go out together (one round trip) instead of
// being interleaved with the arithmetic that consumes them.
template <typename T>
__device__ inline void stage_one(T &v) {
    asm volatile("" : "+v"(v));
}
template <typename... T>
__device__ inline void stage_end(T &...v) {
    (stage_one(v), ...);
}

// Cell of sample i: in LDS, or (CG layout) in the member's slab.
template <bool CG>
__device__ inline int32_t cell_of(const Lds &M, int32_t i) {
    if constexpr (CG) return M.gcell[i];
    else return M.cell[i];
}

// Resolves the proposal of this lane against the member's current state.
// The reads go out in dependent stages; the uniform-mode proposal's reads
// ride along with the first two stages of the guided chain.  GV == 1 is the
// common shape compiled for one EDP shard (G == 1) with a power-of-two slot
// count D, one attention stage (S == 1), 32-bit layer sums, a power-of-two
// score scale and no step log; GV == 0 takes all of these from the arguments.
// RV is the number of row-shards per lane (2 for 65 to 128 row-shards).
template <int DV, int GV, int RV, bool CG, bool HP = false>
__device__ inline Screen screen(const AnnealArgs &a, const Lds &M, const Tables &tb, uint64_t w0, uint64_t w1,
                                uint64_t w2, uint64_t w3, uint64_t w4, uint64_t w5, uint64_t w6, int64_t s1,
                                int64_t s2) {
    Screen sc;
    const int32_t N = a.N, B = a.B, RG = a.RG, D = a.D, G = GV == 1 ? 1 : a.G;
    const bool guided = (uint32_t)w0 < a.p_guide;
    const bool reloc = (uint32_t)(w0 >> 32) < a.rho;
    // Uniform-mode samples (and target cell of a relocation) straight from
    // the words (N, B < 2^16).
    const int32_t ir = (int32_t)bounded_small(w1, (uint32_t)N);
    const int32_t jr = (int32_t)bounded_small(w4, (uint32_t)N);
    const int32_t rc2 = (int32_t)bounded_small(w4, (uint32_t)B);
    // Guided: source row-shard by roulette over J, target over s2 - J_h + 1,
    // whose prefix is V_h = (h + 1)(s2 + 1) - J_pre[h].  Both prefixes are
    // non-decreasing: count the pivots J_pre[8k + 7], then the entries of one
    // block.
    const uint64_t pk1 = bounded_uniform(w1, (uint64_t)s1);
    const uint64_t pk4 = bounded_uniform(w4, (uint64_t)((int64_t)RG * (s2 + 1) - s1));
    // stage 1: pivots; the uniform-mode cells and lengths
    constexpr int NP = 8 * RV;
    int64_t jp[NP], vp[NP];
#pragma unroll
    for (int k = 0; k < NP; ++k) {
        jp[k] = M.Jpiv[k];
        vp[k] = M.Vpiv[k];
    }
    int32_t cir = cell_of<CG>(M, ir), cjr = cell_of<CG>(M, jr);
    int32_t tir = tb.t[ir], tjr = tb.t[jr];
#pragma unroll
    for (int k = 0; k < NP; ++k) stage_end(jp[k], vp[k]);
    stage_end(cir, cjr, tir, tjr);
    int32_t k1 = 0, k4 = 0;
#pragma unroll
    for (int k = 0; k < NP; ++k) {
        k1 += (uint64_t)jp[k] <= pk1 ? 1 : 0;
        k4 += (uint64_t)vp[k] <= pk4 ? 1 : 0;
    }
    k1 = k1 < NP - 1 ? k1 : NP - 1;  // (NP only when s1 == 0, whose pick is redrawn below)
    k4 = k4 < NP - 1 ? k4 : NP - 1;
    const int32_t uc1 = clamp0(cir, B - 1);
    const int32_t uc2 = reloc ? rc2 : clamp0(cjr, B - 1);
    // stage 2: the two blocks; the uniform-mode cell loads and sizes
    int64_t jb[8], vb[8];
#pragma unroll
    for (int x = 0; x < 8; ++x) {
        jb[x] = M.Jpre[8 * k1 + x];
        vb[x] = M.Vpre[8 * k4 + x];
    }
    int32_t uT1 = M.T[uc1], uT2 = M.T[uc2];
    int32_t us0 = M.start[uc1], us1 = M.start[uc1 + 1];
    stage_end(jb[0], jb[1], jb[2], jb[3], jb[4], jb[5], jb[6], jb[7], vb[0], vb[1], vb[2], vb[3], vb[4], vb[5],
              vb[6], vb[7], uT1, uT2, us0, us1);
    int32_t h1 = 8 * k1, h4 = 8 * k4;
#pragma unroll
    for (int x = 0; x < 8; ++x) {
        h1 += (uint64_t)jb[x] <= pk1 ? 1 : 0;
        h4 += (uint64_t)vb[x] <= pk4 ? 1 : 0;
    }
    if (s1 == 0) h1 = (int32_t)bounded_small(w1, (uint32_t)RG);
    h1 = clamp0(h1, RG - 1);
    h4 = clamp0(h4, RG - 1);
    // stage 3: source cell roulette over the row-shard's cell costs (prefix
    // padded with kInf past its slots); target cell uniform over its slots
    int64_t cv[DV];
#pragma unroll
    for (int x = 0; x < DV; ++x) cv[x] = M.Cp[h1 * (DV + 1) + x];
    int64_t tot = M.Ctot[h1];
    int32_t cnt1 = tb.hcnt[h1], cnt2 = tb.hcnt[h4];
    int64_t jlo = M.Jpre[h1 > 0 ? h1 - 1 : 0], jhi = M.Jpre[h1];
    int64_t vlo = M.Vpre[h4 > 0 ? h4 - 1 : 0], vhi = M.Vpre[h4];
    stage_end(tot, cnt1, cnt2, jlo, jhi, vlo, vhi);
    sc.h1 = h1;
    sc.h4 = h4;
    sc.jlo = h1 > 0 ? jlo : 0;
    sc.jhi = jhi;
    sc.vlo = h4 > 0 ? vlo : 0;
    sc.vhi = vhi;
#pragma unroll
    for (int x = 0; x < DV; ++x) stage_end(cv[x]);
    int32_t xi;
    if (tot == 0) {
        xi = (int32_t)bounded_small(w2, (uint32_t)cnt1);
    } else {
        const uint64_t pk2 = __umul64hi(w2, (uint64_t)tot);
        xi = 0;
#pragma unroll
        for (int x = 0; x < DV; ++x) xi += (uint64_t)cv[x] <= pk2 ? 1 : 0;
    }
    xi = clamp0(xi, cnt1 - 1);
    const int32_t x2 = (int32_t)bounded_small(w5, (uint32_t)cnt2);
    int32_t gc1, gc2;
    if (G == 1) {
        gc1 = clamp0(h1 * D + xi, B - 1);
        gc2 = clamp0(h4 * D + x2, B - 1);
    } else {
        gc1 = tb.hcell[h1 * DV + xi];
        gc2 = tb.hcell[h4 * DV + x2];
        stage_end(gc1, gc2);
        gc1 = clamp0(gc1, B - 1);
        gc2 = clamp0(gc2, B - 1);
    }
    // stage 4: member ranges and loads of both cells
    int32_t st1 = M.start[gc1], en1 = M.start[gc1 + 1];
    int32_t st2 = M.start[gc2], en2 = M.start[gc2 + 1];
    int32_t gT1 = M.T[gc1], gT2 = M.T[gc2];
    stage_end(st1, en1, st2, en2, gT1, gT2);
    const int32_t pi = clamp0(st1 + (int32_t)bounded_small(w3, (uint32_t)(en1 - st1)), N - 1);
    const int32_t pj = clamp0(st2 + (int32_t)bounded_small(w6, (uint32_t)(en2 - st2)), N - 1);
    // stage 5: the samples; stage 6: their lengths
    int32_t gi = HP ? M.gpool[pi] : M.pool[pi], gj = HP ? M.gpool[pj] : M.pool[pj];
    stage_end(gi, gj);
    int32_t gti = tb.t[gi], gtj = tb.t[gj];
    stage_end(gti, gtj);
    int32_t c1, c2, T1, T2, sz1, i, j, ti, tj;
    if (guided) {
        c1 = gc1;
        c2 = gc2;
        T1 = gT1;
        T2 = gT2;
        sz1 = en1 - st1;
        i = gi;
        ti = gti;
        sc.pos_i = pi;
        j = reloc ? -1 : gj;
        tj = reloc ? 0 : gtj;
        sc.pos_j = reloc ? -1 : pj;
    } else {
        c1 = uc1;
        c2 = uc2;
        T1 = uT1;
        T2 = uT2;
        sz1 = us1 - us0;
        i = ir;
        ti = tir;
        sc.pos_i = -1;
        j = reloc ? -1 : jr;
        tj = reloc ? 0 : tjr;
        sc.pos_j = -1;
    }
    bool f = c1 != c2;
    if (f) {
        if (!reloc) f = ((int64_t)T1 - ti + tj <= a.C) && ((int64_t)T2 - tj + ti <= a.C);
        else f = (sz1 >= 2) && ((int64_t)T2 + ti <= a.C);
    }
    sc.i = i;
    sc.j = j;
    sc.c1 = c1;
    sc.c2 = c2;
    sc.ti = ti;
    sc.tj = tj;
    sc.feas = f;
    return sc;
}

// #{x in pool[lo, hi) : x < v and x != skip}, uniform over the wave.
__device__ inline int32_t count_less(const uint16_t *pool, int32_t lo, int32_t hi, int32_t v, int32_t skip) {
    int32_t cnt = 0;
    const int lane = lane_id();
    for (int32_t b = lo; b < hi; b += kWave) {
        const int32_t x = b + lane;
        bool pred = false;
        if (x < hi) {
            const int32_t y = pool[x];
            pred = (y < v) && (y != skip);
        }
        cnt += __popcll(__ballot(pred));
    }
    return cnt;
}

// Removes the element at `from` and inserts v at `to`, shifting the elements
// in between by one place, on 32-bit words, four per lane per step.  The
// array is 16-byte aligned and padded by 16 bytes past its last word.
__device__ inline void pool_move(uint16_t *pool16, int32_t from, int32_t to, uint32_t v) {
    uint32_t *pw = reinterpret_cast<uint32_t *>(pool16);
    const int lane = lane_id();
    if (from < to) {
        // new[x] = old[x + 1] for from <= x < to; new[to] = v
        const int32_t wlast = to >> 1;
        for (int32_t base = (from >> 1) & ~3; base <= wlast; base += 4 * kWave) {
            const int32_t w = base + 4 * lane;
            if (w <= wlast) {
                const uint4 c = *reinterpret_cast<const uint4 *>(pw + w);
                const uint32_t nx = pw[w + 4];
                const uint32_t old[4] = {c.x, c.y, c.z, c.w};
                const uint32_t nxt[4] = {c.y, c.z, c.w, nx};
                uint32_t out[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int32_t e0 = 2 * (w + q), e1 = e0 + 1;
                    const uint32_t sh = __builtin_amdgcn_alignbit(nxt[q], old[q], 16);
                    const uint32_t lo = (e0 >= from && e0 < to) ? (sh & 0xFFFFu) : (e0 == to ? v : (old[q] & 0xFFFFu));
                    const uint32_t hi = (e1 >= from && e1 < to) ? (sh >> 16) : (e1 == to ? v : (old[q] >> 16));
                    out[q] = lo | (hi << 16);
                }
                *reinterpret_cast<uint4 *>(pw + w) = make_uint4(out[0], out[1], out[2], out[3]);
            }
            wsync();
        }
    } else if (from > to) {
        // new[x] = old[x - 1] for to < x <= from; new[to] = v (high chunks first)
        const int32_t wfirst = (to >> 1) & ~3;
        for (int32_t top = (from >> 1) & ~3; top >= wfirst; top -= 4 * kWave) {
            const int32_t w = top - 4 * lane;
            if (w >= wfirst) {
                const uint4 c = *reinterpret_cast<const uint4 *>(pw + w);
                const uint32_t pv = w > 0 ? pw[w - 1] : 0u;
                const uint32_t old[4] = {c.x, c.y, c.z, c.w};
                const uint32_t prv[4] = {pv, c.x, c.y, c.z};
                uint32_t out[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int32_t e0 = 2 * (w + q), e1 = e0 + 1;
                    const uint32_t sh = __builtin_amdgcn_alignbit(old[q], prv[q], 16);
                    const uint32_t lo = (e0 > to && e0 <= from) ? (sh & 0xFFFFu) : (e0 == to ? v : (old[q] & 0xFFFFu));
                    const uint32_t hi = (e1 > to && e1 <= from) ? (sh >> 16) : (e1 == to ? v : (old[q] >> 16));
                    out[q] = lo | (hi << 16);
                }
                *reinterpret_cast<uint4 *>(pw + w) = make_uint4(out[0], out[1], out[2], out[3]);
            }
            wsync();
        }
    } else {
        if (lane == 0) pool16[to] = (uint16_t)v;
        wsync();
    }
}

// count_less on an int32 pool in global memory (64 ranks).
__device__ inline int32_t count_less_g(const int32_t *pool, int32_t lo, int32_t hi, int32_t v, int32_t skip) {
    int32_t cnt = 0;
    const int lane = lane_id();
    for (int32_t b = lo; b < hi; b += kWave) {
        const int32_t x = b + lane;
        bool pred = false;
        if (x < hi) {
            const int32_t y = pool[x];
            pred = (y < v) && (y != skip);
        }
        cnt += __popcll(__ballot(pred));
    }
    return cnt;
}

// pool_move on an int32 pool in global memory (64 ranks): each batch loads
// all of its entries before it stores any, and the batches walk in the
// direction of the shift, so no load reads an entry an earlier batch wrote.
// A batch is 2048 entries (32 per lane): a relocation across the pool of the
// largest window shifts up to 32768 entries, one memory round trip a batch.
__device__ inline void pool_move_g(int32_t *pool, int32_t from, int32_t to, int32_t v) {
    const int lane = lane_id();
    constexpr int U = 32;
    if (from < to) {
        // new[x] = old[x + 1] for from <= x < to
        for (int32_t base = from; base < to; base += U * kWave) {
            int32_t val[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t x = base + u * kWave + lane;
                val[u] = x < to ? pool[x + 1] : 0;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t x = base + u * kWave + lane;
                if (x < to) pool[x] = val[u];
            }
        }
    } else if (from > to) {
        // new[x] = old[x - 1] for to < x <= from (high batches first)
        for (int32_t top = from; top > to; top -= U * kWave) {
            int32_t val[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t x = top - u * kWave - lane;
                val[u] = x > to ? pool[x - 1] : 0;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t x = top - u * kWave - lane;
                if (x > to) pool[x] = val[u];
            }
        }
    }
    wsync();
    if (lane == 0) pool[to] = v;
    wsync();
}

// start[c] += d for lo < c <= hi (16-bit entries, 32-bit words four per lane).
__device__ inline void start_add(uint16_t *start16, int32_t lo, int32_t hi, int32_t d) {
    uint32_t *sw = reinterpret_cast<uint32_t *>(start16);
    const int lane = lane_id();
    const int32_t wlast = hi >> 1;
    for (int32_t base = ((lo + 1) >> 1) & ~3; base <= wlast; base += 4 * kWave) {
        const int32_t w = base + 4 * lane;
        if (w <= wlast) {
            const uint4 c = *reinterpret_cast<const uint4 *>(sw + w);
            const uint32_t old[4] = {c.x, c.y, c.z, c.w};
            uint32_t out[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int32_t e0 = 2 * (w + q), e1 = e0 + 1;
                const uint32_t lo16 = (old[q] + ((e0 > lo && e0 <= hi) ? (uint32_t)d : 0u)) & 0xFFFFu;
                const uint32_t hi16 = ((old[q] >> 16) + ((e1 > lo && e1 <= hi) ? (uint32_t)d : 0u)) & 0xFFFFu;
                out[q] = lo16 | (hi16 << 16);
            }
            *reinterpret_cast<uint4 *>(sw + w) = make_uint4(out[0], out[1], out[2], out[3]);
        }
        wsync();
    }
}

// Prefixes of the roulette weights into LDS from J_pre (lane h holds
// J_pre[h], and J_pre[h + 64] in Jp2 when RV == 2): J_pre and
// V_h = (h + 1)(s2 + 1) - J_pre[h], with their pivot entries 8k+7; entries at
// h >= RG hold kInf.
template <int RV>
__device__ inline void write_prefix(const Lds &M, int64_t incl, int64_t incl2, int32_t RG, int64_t s2) {
    const int lane = lane_id();
    const int64_t v = lane < RG ? incl : kInf;
    const int64_t t = lane < RG ? (int64_t)(lane + 1) * (s2 + 1) - incl : kInf;
    M.Jpre[lane] = v;
    M.Vpre[lane] = t;
    if ((lane & 7) == 7) {
        M.Jpiv[lane >> 3] = v;
        M.Vpiv[lane >> 3] = t;
    }
    if (RV == 2) {
        const int32_t h = lane + kWave;
        const int64_t v2 = h < RG ? incl2 : kInf;
        const int64_t t2 = h < RG ? (int64_t)(h + 1) * (s2 + 1) - incl2 : kInf;
        M.Jpre[h] = v2;
        M.Vpre[h] = t2;
        if ((lane & 7) == 7) {
            M.Jpiv[h >> 3] = v2;
            M.Vpiv[h >> 3] = t2;
        }
    }
}

// J_pre of the lane's row-shards (h = lane, and lane + 64 in the second
// value when RV == 2) from their J values.
template <int RV>
__device__ inline void j_prefix(int64_t Jr, int64_t Jr2, int32_t RG, int64_t &incl, int64_t &incl2) {
    const int lane = lane_id();
    incl = wave_incl_scan(lane < RG ? Jr : 0);
    incl2 = RV == 2 ? wave_incl_scan(lane + kWave < RG ? Jr2 : 0) + (int64_t)readlane64((uint64_t)incl, kWave - 1)
                    : 0;
}

template <int RV>
__device__ inline void write_jpre(const Lds &M, int64_t Jr, int64_t Jr2, int32_t RG, int64_t s2) {
    int64_t incl, incl2;
    j_prefix<RV>(Jr, Jr2, RG, incl, incl2);
    write_prefix<RV>(M, incl, incl2, RG, s2);
}

// A row-shard's entry of a lane-distributed table (row-shard h on lane h, or
// on lane h - 64 of the second register when RV == 2); h is wave-uniform.
template <int RV>
__device__ inline int64_t row_entry(int64_t v, int64_t v2, int32_t h) {
    if (RV == 1 || h < kWave) return (int64_t)readlane64((uint64_t)v, h);
    return (int64_t)readlane64((uint64_t)v2, h - kWave);
}

// Member state kept in registers between proposals: J and A of the
// row-shard held by each lane, U of the EDP shard held by each lane, and the
// current score.
struct Regs {
    int64_t Jr, Ar, Ur, s0, s1, s2;
    int64_t Jr2, Ar2;  // row-shards 64..127 (more than 64 row-shards only)
};

// Member slab sections in HBM.
struct SlabPtrs {
    int32_t *cell, *pool, *start, *W;
    int64_t *T, *Q, *J, *A;
};

__device__ inline SlabPtrs slab_ptrs(const AnnealArgs &a, char *slab) {
    SlabPtrs g;
    g.cell = at<int32_t>(slab, a.off.cell);
    g.pool = at<int32_t>(slab, a.off.pool);
    g.start = at<int32_t>(slab, a.off.start);
    g.T = at<int64_t>(slab, a.off.T);
    g.Q = at<int64_t>(slab, a.off.Q);
    g.W = at<int32_t>(slab, a.off.W);
    g.J = at<int64_t>(slab, a.off.J);
    g.A = at<int64_t>(slab, a.off.A);
    return g;
}

// Workgroup tables in LDS: the slot list, slot count and first cost-prefix
// index of every EDP shard, the shard of every slot, the slot count and slot
// cells of every row-shard, and the lengths.
// Every thread of the workgroup takes part (ends with a block barrier).
// CG (the layout with the cell array and lengths in HBM) is a compile-time
// choice so that the lengths pointer is known to be in LDS otherwise: a
// pointer that may be either is read with flat loads, whose waits also wait
// for every outstanding global store (a commit's W rows) before a screen.
template <bool CG>
__device__ inline Tables load_tables(const AnnealArgs &a, char *smem) {
    const int32_t N = a.N, D = a.D, G = a.G;
    int32_t *s_slots = reinterpret_cast<int32_t *>(smem);
    int32_t *s_count = s_slots + G * D;
    int32_t *s_shard = s_count + G;
    int32_t *s_soff = s_shard + D;
    int32_t *s_t = reinterpret_cast<int32_t *>(smem + a.o_tshared);
    for (int32_t x = threadIdx.x; x < G * D; x += blockDim.x) s_slots[x] = a.slots[x];
    for (int32_t x = threadIdx.x; x < G; x += blockDim.x) s_count[x] = a.count[x];
    for (int32_t x = threadIdx.x; x < D; x += blockDim.x) s_shard[x] = a.slot_shard[x];
    if (threadIdx.x == 0) {
        int32_t acc = 0;
        for (int32_t g = 0; g < G; ++g) {
            s_soff[g] = acc;
            acc += a.count[g];
        }
    }
    const int32_t RG = a.RG, DVr = a.dv;
    int32_t *s_hcnt = reinterpret_cast<int32_t *>(smem + a.o_hcnt);
    int32_t *s_hcell = reinterpret_cast<int32_t *>(smem + a.o_hcell);
    // (hq layout with one EDP shard: no slot table, a row-shard's cells are
    // h D + x)
    const bool hcell = !(a.hq && G == 1);
    for (int32_t x = threadIdx.x; x < RG * DVr; x += blockDim.x) {
        const int32_t h = x / DVr, k = x - h * DVr, r = h / G, g = h - r * G, cnt = a.count[g];
        if (k == 0) s_hcnt[h] = cnt;
        if (hcell) s_hcell[x] = r * D + a.slots[g * D + (k < cnt ? k : cnt - 1)];
    }
    if constexpr (CG) {  // the lengths are read from HBM (L2)
        __syncthreads();
        return Tables{s_slots, s_count, s_shard, s_soff, a.t, s_hcnt, s_hcell};
    }
    const int32_t n4 = N >> 2;
    const int4 *t4 = reinterpret_cast<const int4 *>(a.t);
    for (int32_t x = threadIdx.x; x < n4; x += blockDim.x) reinterpret_cast<int4 *>(s_t)[x] = t4[x];
    for (int32_t x = (n4 << 2) + threadIdx.x; x < N; x += blockDim.x) s_t[x] = a.t[x];
    __syncthreads();
    return Tables{s_slots, s_count, s_shard, s_soff, s_t, s_hcnt, s_hcell};
}

__device__ inline Lds member_lds(const AnnealArgs &a, char *smem, int wv) {
    char *mine = smem + a.lds_shared + (int64_t)wv * a.lds_member;
    Lds M;
    M.cell = reinterpret_cast<uint16_t *>(mine + a.o_cell);
    M.pool = reinterpret_cast<uint16_t *>(mine + a.o_pool);
    M.start = reinterpret_cast<uint16_t *>(mine + a.o_start);
    M.T = reinterpret_cast<int32_t *>(mine + a.o_T);
    M.Q = reinterpret_cast<int64_t *>(mine + a.o_Q);
    M.Cp = reinterpret_cast<int64_t *>(mine + a.o_acost);
    M.Ctot = M.Cp + a.RG * (a.dv + 1);
    M.Jpre = reinterpret_cast<int64_t *>(mine + a.o_Jpre);
    M.Vpre = M.Jpre + 64 * a.rv;
    M.Jpiv = M.Jpre + 128 * a.rv;
    M.Vpiv = M.Jpiv + 8 * a.rv;
    return M;
}

// A member's state from a slab into LDS and registers (one wave).  The
// global loads go out in batches of 16 per lane per array before any LDS
// store, so a reload costs few memory round trips.
template <int RV, bool HQ = false>
__device__ inline void member_load(const AnnealArgs &a, const Lds &M, const Tables &tb, const SlabPtrs &g,
                                   Regs &R) {
    const int lane = lane_id();
    const int32_t N = a.N, B = a.B, RG = a.RG, G = a.G;
    constexpr int U = 16;
    if (!(HQ && a.cg)) {  // (64 ranks: the cell array and the pool stay in the slab)
        const int32_t n4 = N >> 2;
        const int4 *c4 = reinterpret_cast<const int4 *>(g.cell), *p4 = reinterpret_cast<const int4 *>(g.pool);
        ushort4 *lc4 = reinterpret_cast<ushort4 *>(M.cell), *lp4 = reinterpret_cast<ushort4 *>(M.pool);
        for (int32_t base = 0; base < n4; base += U * kWave) {
            int4 cu[U], pu[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t x = base + u * kWave + lane;
                if (x < n4) {
                    if (!a.cg) cu[u] = c4[x];  // (CG layout: the cell array stays in the slab)
                    pu[u] = p4[x];
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t x = base + u * kWave + lane;
                if (x < n4) {
                    if (!a.cg)
                        lc4[x] = make_ushort4((uint16_t)cu[u].x, (uint16_t)cu[u].y, (uint16_t)cu[u].z,
                                              (uint16_t)cu[u].w);
                    lp4[x] = make_ushort4((uint16_t)pu[u].x, (uint16_t)pu[u].y, (uint16_t)pu[u].z, (uint16_t)pu[u].w);
                }
            }
        }
        for (int32_t x = (n4 << 2) + lane; x < N; x += kWave) {
            if (!a.cg) M.cell[x] = (uint16_t)g.cell[x];
            M.pool[x] = (uint16_t)g.pool[x];
        }
    }
    for (int32_t base = 0; base <= B; base += U * kWave) {
        int32_t sv[U];
        int64_t tv[U], qv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int32_t x = base + u * kWave + lane;
            if (x <= B) sv[u] = g.start[x];
            if (x < B) {
                tv[u] = g.T[x];
                if (!HQ) qv[u] = g.Q[x];  // (HQ: Q is used in place in the slab)
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int32_t x = base + u * kWave + lane;
            if (x <= B) M.start[x] = (uint16_t)sv[u];
            if (x < B) {
                M.T[x] = (int32_t)tv[u];
                if (!HQ) M.Q[x] = qv[u];
            }
        }
    }
    const int32_t h2 = lane + kWave;  // the lane's second row-shard (more than 64 only)
    R.Jr = lane < RG ? g.J[lane] : 0;
    R.Ar = lane < RG ? g.A[lane] : 0;
    R.Jr2 = RV == 2 && h2 < RG ? g.J[h2] : 0;
    R.Ar2 = RV == 2 && h2 < RG ? g.A[h2] : 0;
    wsync();
    // cost prefix of each row-shard's cells, in slot order (lanes over row-shards)
    for (int32_t h = lane; h < (RV == 2 ? RG : (RG < kWave ? RG : kWave)); h += kWave) {
        const int32_t cnt = tb.hcnt[h];
        int64_t acc = 0;
        int64_t *cp = M.Cp + h * (a.dv + 1);
        for (int32_t x = 0; x < a.dv; ++x) {
            if (x < cnt) {
                const int32_t c = HQ && G == 1 ? h * a.D + x : tb.hcell[h * a.dv + x];
                const int64_t t = M.T[c], q = M.Q[c];
                for (int s = 0; s < a.S; ++s) acc += a.alpha[s] * t + a.beta[s] * q;
                cp[x] = acc;
            } else {
                cp[x] = kInf;
            }
        }
        M.Ctot[h] = acc;
    }
    // U_g = sum over rows of J(r, g); lane g holds it
    int64_t Ur = 0;
    const int32_t gl = lane - (lane / G) * G, gl2 = h2 - (h2 / G) * G;
    for (int32_t gg = 0; gg < G; ++gg) {
        const int64_t u = wave_sum((lane < RG && gl == gg ? R.Jr : 0) + (RV == 2 && h2 < RG && gl2 == gg ? R.Jr2 : 0));
        if (lane == gg) Ur = u;
    }
    R.Ur = Ur;
    R.s0 = wave_max(lane < G ? Ur : LLONG_MIN);
    R.s1 = wave_sum(lane < G ? Ur : 0);
    const int64_t j1 = lane < RG ? R.Jr : LLONG_MIN, j2 = RV == 2 && h2 < RG ? R.Jr2 : LLONG_MIN;
    R.s2 = wave_max(j1 > j2 ? j1 : j2);
    write_jpre<RV>(M, R.Jr, R.Jr2, RG, R.s2);
    wsync();
}

// A member's state back to a slab (W is kept up to date in the slab, and Q
// too with HQ).
template <int RV, bool HQ = false>
__device__ inline void member_store(const AnnealArgs &a, const Lds &M, const SlabPtrs &g, const Regs &R) {
    const int lane = lane_id();
    const int32_t N = a.N, B = a.B, RG = a.RG;
    wsync();
    const int32_t n4 = N >> 2;
    int4 *c4 = reinterpret_cast<int4 *>(g.cell), *p4 = reinterpret_cast<int4 *>(g.pool);
    const ushort4 *lc4 = reinterpret_cast<const ushort4 *>(M.cell), *lp4 = reinterpret_cast<const ushort4 *>(M.pool);
    if (!(HQ && a.cg)) {  // (64 ranks: the slab's cell array and pool are already current)
        for (int32_t x = lane; x < n4; x += kWave) {
            const ushort4 v = lp4[x];
            if (!a.cg) {  // (CG layout: the slab's cell array is already current)
                const ushort4 u = lc4[x];
                c4[x] = make_int4(u.x, u.y, u.z, u.w);
            }
            p4[x] = make_int4(v.x, v.y, v.z, v.w);
        }
        for (int32_t x = (n4 << 2) + lane; x < N; x += kWave) {
            if (!a.cg) g.cell[x] = M.cell[x];
            g.pool[x] = M.pool[x];
        }
    }
    for (int32_t x = lane; x <= B; x += kWave) g.start[x] = M.start[x];
    for (int32_t x = lane; x < B; x += kWave) {
        g.T[x] = M.T[x];
        if (!HQ) g.Q[x] = M.Q[x];
    }
    if (lane < RG) {
        g.J[lane] = R.Jr;
        g.A[lane] = R.Ar;
    }
    if (RV == 2 && lane + kWave < RG) {
        g.J[lane + kWave] = R.Jr2;
        g.A[lane + kWave] = R.Ar2;
    }
}

// One level (K proposals) of member m from its current state, at the given
// level index and temperature; x0..x2 is the incumbent score at the level
// start.  Writes the member's result row.
// Summary of a member's level for the level end.
struct LevelOut {
    int64_t b0, b1, b2;  // trajectory best
    double e;            // terminal energy
};

// GV selects the variant: 1 the common shape (see screen), 0 the general
// one, 2 the general one with two row-shards per lane (65 to 128).  LV is
// the number of layers per lane (2 for 33 to 64 layers).
template <int PV, int DV, int GV, int LV, bool CG>
__device__ inline LevelOut member_level(const AnnealArgs &a, const Lds &M, const Tables &tb, int32_t *W, int m,
                                        int32_t level, double temp, int64_t x0, int64_t x1, int64_t x2,
                                        uint8_t *log_arg, int64_t *res, int64_t *trace_row, Regs &R) {
    constexpr int RV = GV == 2 ? 2 : 1;
    constexpr bool HP = PV == 64;  // (64 ranks: the pool is in the slab)
    uint8_t *const log = GV == 1 ? nullptr : log_arg;  // (the common shape is launched without a step log)
    const int lane = lane_id();
    const int32_t N = a.N, B = a.B, RG = a.RG, D = a.D, G = GV == 1 ? 1 : a.G, L = a.L;
    int64_t Jr = R.Jr, Ar = R.Ar, Ur = R.Ur, s0 = R.s0, s1 = R.s1, s2 = R.s2;
    int64_t Jr2 = RV == 2 ? R.Jr2 : 0, Ar2 = RV == 2 ? R.Ar2 : 0;  // row-shards 64..127
    // J_pre of the lane's row-shards, kept up to date by each move's J deltas
    int64_t Jp, Jp2;
    j_prefix<RV>(Jr, Jr2, RG, Jp, Jp2);
    int64_t b0 = s0, b1 = s1, b2 = s2;
    int32_t best_is_start = 1;
    int32_t *bl = a.best + (int64_t)m * N;
    if (lex_less(s0, s1, s2, x0, x1, x2)) {
        // A start state better than the incumbent is itself a trajectory
        // best; keep its layout, since the state is updated in place.
        for (int32_t x = lane; x < N; x += kWave) bl[x] = cell_of<CG>(M, x);
        best_is_start = 0;
    }
    int64_t n_acc = 0, n_eval = 0;
    double e_cur = GV == 1 ? energy_pow2(a, s0, s1, s2) : energy_k(a, s0, s1, s2);
    const int half = lane >> 5, hl = lane & 31;
    // cells of a row-shard: lane (half, x) holds its x-th slot, x < 16 (all
    // 32 lanes of the half with up to 32 slots)
    const int cx = DV > 16 ? hl : (lane & 15);
    const bool cell_lane = DV > 16 || (lane & 16) == 0;
    // layer v of the lane is hl + 32 v (v < LV), held when below L
    auto lay_act = [&](int v) { return hl + 32 * v < L; };
    // Loads of one move: lane (half, hl) reads its layers of row-shard ha
    // (half 0) or hb (half 1), the q row that leaves that row-shard (qx) and
    // the one that enters it (qy), so every lane's new row is wr - qx + qy.
    // A relocation moves no sample back: its missing row is the zero row.
    // Rows are chunk-major ([P/4][L][4]): chunk x of layer ll is int4 x * L + ll.
    // Entry v * PV / 4 + x of wr, qx, qy is chunk x of the lane's layer v.
    auto load_rows = [&](int32_t i, int32_t j, int32_t ha, int32_t hb, int4 *wr, int4 *qx, int4 *qy) {
        const int32_t row = half ? hb : ha;
        const int32_t *qi = a.qt + (int64_t)i * a.LP, *qj = j >= 0 ? a.qt + (int64_t)j * a.LP : a.qzero;
#pragma unroll
        for (int v = 0; v < LV; ++v) {
            const int32_t ll = lay_act(v) ? hl + 32 * v : L - 1;
            const int4 *wp = reinterpret_cast<const int4 *>(W + (int64_t)row * a.LP) + ll;
            const int4 *xp = reinterpret_cast<const int4 *>(half ? qj : qi) + ll;
            const int4 *yp = reinterpret_cast<const int4 *>(half ? qi : qj) + ll;
#pragma unroll
            for (int x = 0; x < PV / 4; ++x) {
                wr[v * (PV / 4) + x] = wp[x * L];
                qx[v * (PV / 4) + x] = xp[x * L];
                qy[v * (PV / 4) + x] = yp[x * L];
            }
        }
    };

    // 64 ranks: a lane's new row (128 entries with two layers) is formed
    // from the W row and the two q rows 16 ranks at a time, so only one
    // chunk of each is in registers besides the new row.
    auto rows_nw64 = [&](int32_t i, int32_t j, int32_t ha, int32_t hb, int32_t *nw) {
        const int32_t row = half ? hb : ha;
        const int32_t *qi = a.qt + (int64_t)i * a.LP, *qj = j >= 0 ? a.qt + (int64_t)j * a.LP : a.qzero;
        constexpr int CH = 4;  // 16-byte chunks (four ranks each) per pass
#pragma unroll
        for (int c = 0; c < PV / 4; c += CH) {
            int4 w4[LV * CH], x4[LV * CH], y4[LV * CH];
#pragma unroll
            for (int v = 0; v < LV; ++v) {
                const int32_t ll = lay_act(v) ? hl + 32 * v : L - 1;
                const int4 *wp = reinterpret_cast<const int4 *>(W + (int64_t)row * a.LP) + ll;
                const int4 *xp = reinterpret_cast<const int4 *>(half ? qj : qi) + ll;
                const int4 *yp = reinterpret_cast<const int4 *>(half ? qi : qj) + ll;
#pragma unroll
                for (int x = 0; x < CH; ++x) {
                    w4[v * CH + x] = wp[(c + x) * L];
                    x4[v * CH + x] = xp[(c + x) * L];
                    y4[v * CH + x] = yp[(c + x) * L];
                }
            }
#pragma unroll
            for (int v = 0; v < LV; ++v)
#pragma unroll
                for (int x = 0; x < CH; ++x) {
                    const int y = v * PV + 4 * (c + x), u = v * CH + x;
                    nw[y + 0] = w4[u].x - x4[u].x + y4[u].x;
                    nw[y + 1] = w4[u].y - x4[u].y + y4[u].y;
                    nw[y + 2] = w4[u].z - x4[u].z + y4[u].z;
                    nw[y + 3] = w4[u].w - x4[u].w + y4[u].w;
                }
        }
    };

    for (int32_t k0 = 0; k0 < a.K; k0 += kWave) {
        const int32_t k = k0 + lane;
        const U64x4 b0w = philox4x64_10((uint64_t)k, (uint64_t)(uint32_t)level, (uint64_t)(uint32_t)m, 0,
                                        a.seed, 0);
        const U64x4 b1w = philox4x64_10((uint64_t)k, (uint64_t)(uint32_t)level, (uint64_t)(uint32_t)m, 1,
                                        a.seed, 0);
        const uint64_t w0 = b0w.v[0], w1 = b0w.v[1], w2 = b0w.v[2], w3 = b0w.v[3];
        const uint64_t w4 = b1w.v[0], w5 = b1w.v[1], w6 = b1w.v[2], w7 = b1w.v[3];
        uint64_t pending = __ballot(k < a.K);
        Screen sc = screen<DV, GV, RV, CG, HP>(a, M, tb, w0, w1, w2, w3, w4, w5, w6, s1, s2);
        uint64_t feas = __ballot(sc.feas && k < a.K);
        uint64_t valid = ~0ull;  // lanes whose screen is current
        while (pending) {
            uint64_t cand = pending & feas;
            {
                // The next candidate and every pending lane below it must be
                // current; otherwise screen the batch again.
                const uint64_t stale = pending & ~valid;
                if (stale && (!cand || (stale & (~stale + 1)) <= (cand & (~cand + 1)))) {
                    sc = screen<DV, GV, RV, CG, HP>(a, M, tb, w0, w1, w2, w3, w4, w5, w6, s1, s2);
                    feas = __ballot(sc.feas && k < a.K);
                    valid = ~0ull;
                    cand = pending & feas;
                }
            }
            const uint64_t below = cand ? (cand & (~cand + 1)) - 1 : ~0ull;
            if (log && ((pending & below) >> lane) & 1ull) log[k] = 0;
            if (!cand) break;
            const int f = first_lane(cand);
            pending &= ~((cand & (~cand + 1)) | below);
            // ---- evaluate proposal f (uniform)
            const int32_t i = clamp0(__builtin_amdgcn_readlane(sc.i, f), N - 1);
            const int32_t jf = __builtin_amdgcn_readlane(sc.j, f);
            const int32_t j = jf < 0 ? -1 : clamp0(jf, N - 1);
            const int32_t c1 = clamp0(__builtin_amdgcn_readlane(sc.c1, f), B - 1);
            const int32_t c2 = clamp0(__builtin_amdgcn_readlane(sc.c2, f), B - 1);
            int32_t pos_i = __builtin_amdgcn_readlane(sc.pos_i, f);
            int32_t pos_j = __builtin_amdgcn_readlane(sc.pos_j, f);
            const int64_t ti = __builtin_amdgcn_readlane(sc.ti, f);
            const int64_t tj = __builtin_amdgcn_readlane(sc.tj, f);
            const uint32_t fw0 = __builtin_amdgcn_readlane((int32_t)(uint32_t)(w0 >> 32), f);
            const uint32_t fw7 = __builtin_amdgcn_readlane((int32_t)(uint32_t)(w7 >> 32), f);
            const bool reloc = fw0 < a.rho;
            n_eval += 1;
            const int32_t ra = GV == 1 ? c1 >> a.dshift : div_small(c1, D, a.dinv);
            const int32_t rb = GV == 1 ? c2 >> a.dshift : div_small(c2, D, a.dinv);
            const int32_t ga = G == 1 ? 0 : tb.shard[c1 - ra * D], gb = G == 1 ? 0 : tb.shard[c2 - rb * D];
            const int32_t ha = ra * G + ga, hb = rb * G + gb;
            const bool two = ha != hb;
            // W rows of a and b, q rows of i and j: issue the loads first.
            // They are issued (and consumed below) on every path, also when
            // both cells are in one row-shard (the row is then read twice):
            // a load left pending on some path would make the compiler wait
            // on the memory counter, which the previous commit's W stores
            // share, before the next move's loads.
            constexpr int NR = PV <= 32 ? LV * PV / 4 : 1;  // (64 ranks: rows_nw64 below)
            int4 wr[NR], qx[NR], qy[NR];
            if constexpr (PV <= 32) load_rows(i, j, ha, hb, wr, qx, qy);
            // Cell statistics of the two row-shards (lanes (half, cx)) and the
            // commit inputs, read in one stage while the row loads are in
            // flight: the member ranges of both cells and, when both fit 32
            // lanes, their members (half 0: c1, half 1: c2; left in flight
            // until the commit).
            const int32_t hsel = half ? hb : ha;
            int32_t cnt = D, cc = hsel * D + cx;  // (one EDP shard: every row-shard is a row of D slots)
            if (G != 1) {
                cnt = tb.hcnt[hsel];
                cc = tb.hcell[hsel * DV + (cx < DV ? cx : 0)];
                stage_end(cnt, cc);
            }
            const bool cact = cell_lane && cx < cnt && (half == 0 || two);
            int32_t st1 = M.start[c1], en1 = M.start[c1 + 1];
            int32_t st2 = M.start[c2], en2 = M.start[c2 + 1];
            int64_t Tc = 0, Qc = 0;
            if (cact) {
                Tc = M.T[cc];
                Qc = M.Q[cc];
            }
            int64_t T1 = M.T[c1], T2 = M.T[c2], Q1 = M.Q[c1], Q2v = M.Q[c2];
            stage_end(st1, en1, st2, en2, Tc, Qc, T1, T2, Q1, Q2v);
            const int32_t sz1 = en1 - st1, sz2 = en2 - st2;
            const bool small = sz1 <= 32 && sz2 <= 32;
            int32_t y = -1;
            bool yv = false;
            if (small) {
                const int32_t sz = half ? sz2 : sz1;
                yv = hl < sz;
                if (yv) y = HP ? M.gpool[(half ? st2 : st1) + hl] : M.pool[(half ? st2 : st1) + hl];
            }
            if (cact) {
                if (cc == c1) {
                    Tc += tj - ti;
                    Qc += tj * tj - ti * ti;
                }
                if (cc == c2) {  // (never the same cell as c1)
                    Tc += ti - tj;
                    Qc += ti * ti - tj * tj;
                }
            }
            const int64_t nT1 = T1 - ti + tj, nT2 = T2 + ti - tj;
            const int64_t nQ1 = Q1 - ti * ti + tj * tj, nQ2 = Q2v + ti * ti - tj * tj;
            int64_t Arow = 0, cw = 0;
#pragma unroll
            for (int s = 0; s < kMaxStages; ++s) {
                if (s < (GV == 1 ? 1 : a.S)) {
                    const int64_t cost = a.alpha[s] * Tc + a.beta[s] * Qc;
                    cw += cact ? cost : 0;
                    Arow = (int64_t)((uint64_t)Arow + (uint64_t)row_head_max64<DV>(cact ? cost : LLONG_MIN));
                }
            }
            const int64_t Aa = (int64_t)readlane64((uint64_t)Arow, DV > 16 ? 16 : 0);
            const int64_t Ab = two ? (int64_t)readlane64((uint64_t)Arow, DV > 16 ? 48 : 32) : Aa;
            const int64_t Jha = row_entry<RV>(Jr, Jr2, ha), Aha = row_entry<RV>(Ar, Ar2, ha);
            const int64_t Jhb = row_entry<RV>(Jr, Jr2, hb);
            int64_t Ja, Jb;
            int32_t nw[LV * PV];
            if constexpr (PV <= 32) {
#pragma unroll
                for (int x = 0; x < LV * PV / 4; ++x) {
                    nw[4 * x + 0] = wr[x].x - qx[x].x + qy[x].x;
                    nw[4 * x + 1] = wr[x].y - qx[x].y + qy[x].y;
                    nw[4 * x + 2] = wr[x].z - qx[x].z + qy[x].z;
                    nw[4 * x + 3] = wr[x].w - qx[x].w + qy[x].w;
                }
            } else {
                rows_nw64(i, j, ha, hb, nw);
            }
            if (two) {
                // the lane's share of the layer sum: the rank maximum of each
                // of its layers (at most L W_b < 2^31 in the 32-bit case)
                int32_t mx32 = 0;
                int64_t mx64 = 0;
#pragma unroll
                for (int v = 0; v < LV; ++v) {
                    int32_t mx = INT32_MIN;
#pragma unroll
                    for (int p = 0; p < PV; ++p) mx = nw[v * PV + p] > mx ? nw[v * PV + p] : mx;
                    mx32 += lay_act(v) ? mx : 0;
                    mx64 += lay_act(v) ? (int64_t)mx : 0;
                }
                int64_t suma, sumb;
                if (GV == 1 || a.sum32) {  // L times the W bound fits 31 bits
                    const int32_t sm = row_sum32(mx32);
                    suma = (int64_t)__builtin_amdgcn_readlane(sm, 0) + __builtin_amdgcn_readlane(sm, 16);
                    sumb = (int64_t)__builtin_amdgcn_readlane(sm, 32) + __builtin_amdgcn_readlane(sm, 48);
                } else {
                    const int64_t sm = row_sum64(mx64);
                    suma = (int64_t)(readlane64((uint64_t)sm, 0) + readlane64((uint64_t)sm, 16));
                    sumb = (int64_t)(readlane64((uint64_t)sm, 32) + readlane64((uint64_t)sm, 48));
                }
                Ja = Aa + (suma << a.F);
                Jb = Ab + (sumb << a.F);
            } else {
                Ja = Aa + (Jha - Aha);  // (nw unused: W does not change)
                Jb = Ja;
            }
            const int64_t dJa = Ja - Jha, dJb = two ? Jb - Jhb : 0;
            const int64_t n1 = s1 + dJa + dJb;
            int64_t n0, Un = Ur;
            if (G == 1) {
                n0 = n1;
                Un = n1;
            } else {
                if (lane == ga) Un += dJa;
                if (lane == gb && two) Un += dJb;
                // the maximum of the other shards is s0 unless ga or gb held it
                const int64_t Uga = (int64_t)readlane64((uint64_t)Ur, ga), Ugb = (int64_t)readlane64((uint64_t)Ur, gb);
                if (Uga < s0 && Ugb < s0) {
                    if (gb == ga) {
                        const int64_t na = Uga + dJa + dJb;
                        n0 = s0 > na ? s0 : na;
                    } else {
                        const int64_t na = Uga + dJa, nb = Ugb + dJb;
                        n0 = s0 > na ? s0 : na;
                        n0 = n0 > nb ? n0 : nb;
                    }
                } else {
                    n0 = wave_max(lane < G ? Un : LLONG_MIN);
                }
            }
            // the maximum of the other row-shards is s2 unless ha or hb held it
            int64_t n2;
            if (Jha < s2 && Jhb < s2) {
                n2 = s2 > Ja ? s2 : Ja;
                n2 = n2 > Jb ? n2 : Jb;
            } else {
                const int64_t Jn = lane == ha ? Ja : (lane == hb ? Jb : Jr);
                int64_t mx = lane < RG ? Jn : LLONG_MIN;
                if (RV == 2) {
                    const int32_t h2 = lane + kWave;
                    const int64_t Jn2 = h2 == ha ? Ja : (h2 == hb ? Jb : Jr2);
                    mx = h2 < RG && Jn2 > mx ? Jn2 : mx;
                }
                n2 = wave_max(mx);
            }
            const double e_new = GV == 1 ? energy_pow2(a, n0, n1, n2) : energy_k(a, n0, n1, n2);
            bool accept = lex_less(n0, n1, n2, s0, s1, s2);
            if (!accept && !(e_new > e_cur)) accept = true;  // delta <= 0 (the divisor is >= 1)
            if (!accept) {
                const double den = fabs(e_cur) > 1.0 ? fabs(e_cur) : 1.0;
                const double delta = (e_new - e_cur) / den;
                if (!(delta > 0.0)) {
                    accept = true;  // z = 0 and exp(0) = 1 > u
                } else {
                    const double z = delta / temp;
                    const double u = (double)fw7 * (1.0 / 4294967296.0);
                    // u < exp_det(-z), decided without the series when u is
                    // clear of the bracket 1 - z <= exp(-z) <= 1 - z + z^2/2
                    // (z >= 0); the 2^-40 margins exceed every rounding error
                    // of the bounds and of exp_det (a few ulp).
                    const double omz = 1.0 - z;
                    if (z < 0.5 && u < omz * (1.0 - 0x1p-40)) accept = true;
                    else if (z < 0.5 && u >= (omz + (0.5 * z) * z) * (1.0 + 0x1p-40)) accept = false;
                    else accept = u < exp_det(-z);
                }
            }
            if (!accept) {
                if (log && lane == f) log[k] = 1;
                continue;  // the remaining screens stay valid
            }
            if (log && lane == f) log[k] = 2;
            n_acc += 1;
            // ---- commit
            wsync();
            if (two) {
#pragma unroll
                for (int v = 0; v < LV; ++v) {
                    if (!lay_act(v)) continue;
                    int4 *wp = reinterpret_cast<int4 *>(W + (int64_t)(half ? hb : ha) * a.LP) + hl + 32 * v;
#pragma unroll
                    for (int x = 0; x < PV / 4; ++x) {
                        const int y = v * PV + 4 * x;
                        wp[x * L] = make_int4(nw[y], nw[y + 1], nw[y + 2], nw[y + 3]);
                    }
                }
            }
            if (!reloc) {
                if (small) {
                    // half 0: cell c1 drops i, takes j; half 1: cell c2 drops j, takes i
                    const int32_t out = half ? j : i, in = half ? i : j;
                    const uint64_t lt = __ballot(yv && y != out && y < in);
                    const int32_t pin = __popcll(lt & (half ? 0xFFFFFFFF00000000ull : 0xFFFFFFFFull));
                    const int32_t st = half ? st2 : st1;
                    if (yv) {
                        const int32_t at = y == out ? st + pin : st + hl - (out < y ? 1 : 0) + (in < y ? 1 : 0);
                        const int32_t val = y == out ? in : y;
                        if constexpr (HP) M.gpool[at] = val;
                        else M.pool[at] = (uint16_t)val;
                    }
                    wsync();
                } else {
                    auto cl = [&](int32_t lo, int32_t hi, int32_t v, int32_t skip) {
                        return HP ? count_less_g(M.gpool, lo, hi, v, skip) : count_less(M.pool, lo, hi, v, skip);
                    };
                    auto mv = [&](int32_t from, int32_t to, int32_t v) {
                        if constexpr (HP) pool_move_g(M.gpool, from, to, v);
                        else pool_move(M.pool, from, to, (uint32_t)v);
                    };
                    if (pos_i < 0) pos_i = st1 + cl(st1, en1, i, -1);
                    if (pos_j < 0) pos_j = st2 + cl(st2, en2, j, -1);
                    const int32_t to1 = st1 + cl(st1, en1, j, i);
                    const int32_t to2 = st2 + cl(st2, en2, i, j);
                    wsync();
                    mv(clamp0(pos_i, N - 1), clamp0(to1, N - 1), j);
                    mv(clamp0(pos_j, N - 1), clamp0(to2, N - 1), i);
                }
            } else {
                int32_t rk;
                if (small) {
                    const uint64_t b1 = __ballot(yv && half == 0 && y < i);
                    const uint64_t b2 = __ballot(yv && half == 1 && y < i);
                    if (pos_i < 0) pos_i = st1 + __popcll(b1);
                    rk = __popcll(b2);
                } else {
                    if (pos_i < 0)
                        pos_i = st1 + (HP ? count_less_g(M.gpool, st1, en1, i, -1) : count_less(M.pool, st1, en1, i, -1));
                    rk = HP ? count_less_g(M.gpool, st2, en2, i, -1) : count_less(M.pool, st2, en2, i, -1);
                }
                const int32_t to = c1 < c2 ? st2 - 1 + rk : st2 + rk;
                wsync();
                if constexpr (HP) pool_move_g(M.gpool, clamp0(pos_i, N - 1), clamp0(to, N - 1), i);
                else pool_move(M.pool, clamp0(pos_i, N - 1), clamp0(to, N - 1), (uint32_t)i);
                if (c1 < c2) start_add(M.start, c1, c2, -1);
                else start_add(M.start, c2, c1, 1);
            }
            if (lane == 0) {
                if constexpr (CG) {
                    M.gcell[i] = c2;
                    if (j >= 0) M.gcell[j] = c1;
                } else {
                    M.cell[i] = (uint16_t)c2;
                    if (j >= 0) M.cell[j] = (uint16_t)c1;
                }
                M.T[c1] = (int32_t)nT1;
                M.Q[c1] = nQ1;
                M.T[c2] = (int32_t)nT2;
                M.Q[c2] = nQ2;
            }
            {
                const int64_t incl = row_incl_scan64<DV>(cw);
                if (cact) M.Cp[hsel * (DV + 1) + cx] = incl;
                if (cact && cx == cnt - 1) M.Ctot[hsel] = incl;
            }
            if (lane == ha) {
                Jr = Ja;
                Ar = Aa;
            } else if (lane == hb) {
                Jr = Jb;
                Ar = Ab;
            }
            if (RV == 2) {
                if (lane + kWave == ha) {
                    Jr2 = Ja;
                    Ar2 = Aa;
                } else if (lane + kWave == hb) {
                    Jr2 = Jb;
                    Ar2 = Ab;
                }
            }
            // J_pre moves by dJa from row-shard ha on and by dJb from hb on
            auto shift = [&](int32_t h) -> int64_t { return (h >= ha ? dJa : 0) + (h >= hb ? dJb : 0); };
            Jp += shift(lane);
            if (RV == 2) Jp2 += shift(lane + kWave);
            write_prefix<RV>(M, Jp, Jp2, RG, n2);
            if (pending) {
                // A screen stays current unless the move touched what it
                // read: its cells (lengths, members, sizes), the cell costs
                // of its source row-shard, or the prefix interval holding
                // one of its picks.  A pick keeps its row-shard when it lies
                // in the interval after the move's J deltas; V_pre moves by
                // (h + 1)(n2 - s2) besides.  A relocation shifts the members
                // of the cells strictly between its two cells by one place.
                const int64_t ds2 = n2 - s2;
                sc.jlo += shift(sc.h1 - 1);
                sc.jhi += shift(sc.h1);
                sc.vlo += (int64_t)sc.h4 * ds2 - shift(sc.h4 - 1);
                sc.vhi += (int64_t)(sc.h4 + 1) * ds2 - shift(sc.h4);
                bool keep = sc.c1 != c1 && sc.c1 != c2 && sc.c2 != c1 && sc.c2 != c2;
                if ((uint32_t)w0 < a.p_guide) {
                    const uint64_t pk1 = bounded_uniform(w1, (uint64_t)n1);
                    const uint64_t pk4 = bounded_uniform(w4, (uint64_t)((int64_t)RG * (n2 + 1) - n1));
                    keep = keep && sc.h1 != ha && sc.h1 != hb && (uint64_t)sc.jlo <= pk1 &&
                           pk1 < (uint64_t)sc.jhi && (uint64_t)sc.vlo <= pk4 && pk4 < (uint64_t)sc.vhi;
                }
                if (reloc) {
                    const int32_t lo = c1 < c2 ? c1 : c2, hi = c1 < c2 ? c2 : c1, d = c1 < c2 ? -1 : 1;
                    if (sc.pos_i >= 0 && sc.c1 > lo && sc.c1 < hi) sc.pos_i += d;
                    if (sc.pos_j >= 0 && sc.c2 > lo && sc.c2 < hi) sc.pos_j += d;
                }
                // (screens drawn while s1 was 0 picked h1 uniformly)
                valid = s1 > 0 && n1 > 0 ? valid & __ballot(keep) : 0;
            }
            Ur = Un;
            s0 = n0;
            s1 = n1;
            s2 = n2;
            e_cur = e_new;
            wsync();
            if (lex_less(s0, s1, s2, b0, b1, b2)) {
                b0 = s0;
                b1 = s1;
                b2 = s2;
                best_is_start = 0;
                if (lex_less(s0, s1, s2, x0, x1, x2))
                    for (int32_t x = lane; x < N; x += kWave) bl[x] = cell_of<CG>(M, x);
            }
        }
    }
    R.Jr = Jr;
    R.Ar = Ar;
    if (RV == 2) {
        R.Jr2 = Jr2;
        R.Ar2 = Ar2;
    }
    R.Ur = Ur;
    R.s0 = s0;
    R.s1 = s1;
    R.s2 = s2;
    if (lane == 0) {
        res[0] = s0; res[1] = s1; res[2] = s2;
        res[3] = b0; res[4] = b1; res[5] = b2;
        res[6] = n_acc; res[7] = n_eval;
        res[8] = best_is_start;
        res[9] = m;
        if (trace_row) {
            trace_row[0] = s0; trace_row[1] = s1; trace_row[2] = s2;
            trace_row[3] = b0; trace_row[4] = b1; trace_row[5] = b2;
            trace_row[6] = n_acc; trace_row[7] = n_eval;
        }
    }
    return LevelOut{b0, b1, b2, e_cur};
}

}  // namespace

// Members per workgroup of the chain kernels (one wave each): four waves
// leave every wave the whole register file of its SIMD.
constexpr int kRunMaxWaves = 4;

// One level of every member: state from the member's slab, K proposals,
// state back to the slab.
template <int PV, int DV, int GV, int LV, bool CG>
__global__ void __launch_bounds__(kRunMaxWaves * kWave) k_anneal_chain(AnnealArgs a) {
    extern __shared__ __align__(16) char smem[];
    const Tables tb = load_tables<CG>(a, smem);
    const int wv = wave_id();
    const int m = blockIdx.x * a.mpw + wv;
    if (m >= a.pop) return;  // no block barrier follows
    Lds M = member_lds(a, smem, wv);
    const SlabPtrs g = slab_ptrs(a, a.slabs + (int64_t)a.slab_of[m] * a.off.bytes);
    M.gcell = g.cell;
    constexpr bool HQ = PV == 64;  // (64 ranks: the hq layout)
    if constexpr (HQ) {
        M.gpool = g.pool;
        M.Q = g.Q;
        M.Cp = a.gcp + (int64_t)m * a.cp_stride;
        M.Ctot = M.Cp + a.RG * (a.dv + 1);
    }
    Regs R;
    member_load<GV == 2 ? 2 : 1, HQ>(a, M, tb, g, R);
    member_level<PV, DV, GV, LV, CG>(a, M, tb, g.W, m, a.level, a.temp, a.xscore[0], a.xscore[1], a.xscore[2],
                         a.step_log ? a.step_log + (int64_t)m * a.K : nullptr, a.results + (int64_t)m * kRes,
                         nullptr, R);
    member_store<GV == 2 ? 2 : 1, HQ>(a, M, g, R);
}

// ---------------------------------------------------------------------------
// Whole schedule in one cooperative launch.  Every workgroup stays resident;
// a wave keeps its member's state in LDS and registers from level to level.
// Wave gw owns slab gw for the whole run; the member it runs changes with
// resampling.  After a level, every workgroup computes the same level end
// from the members' result rows: the incumbent update, the systematic
// resampling parents, and the slab hand-over (the first child of a parent
// keeps the parent's wave and slab; every further child takes the wave of a
// member without children, which reloads the parent's published state).
// Grid barriers: A after the results, B after publishing parent states, C
// after the copies (only when there are copies).

namespace {

// Hand-over of a member to another wave through global memory: the raw LDS
// region (16-byte units, all reads then all writes per batch) and the
// registers.  Every lane of the wave takes part.
typedef int32_t v4i __attribute__((ext_vector_type(4)));
// Copies n 16-byte units from src to dst with one wave, 16 loads per lane in
// flight before the stores.
__device__ inline void wave_copy16(const char *src, char *dst, int32_t n) {
    const v4i *s4 = reinterpret_cast<const v4i *>(src);
    v4i *d4 = reinterpret_cast<v4i *>(dst);
    const int lane = lane_id();
    constexpr int U = 16;
    for (int32_t base = 0; base < n; base += U * kWave) {
        v4i v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int32_t x = base + u * kWave + lane;
            v[u] = s4[x < n ? x : n - 1];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int32_t x = base + u * kWave + lane;
            if (x < n) d4[x] = v[u];
        }
    }
}

template <int RV>
__device__ inline void member_publish(const AnnealArgs &a, const char *mine, char *blob, const Regs &R) {
    const int lane = lane_id();
    wsync();
    const int32_t n16 = a.lds_member >> 4;
    const v4i *src = reinterpret_cast<const v4i *>(mine);
    v4i *dst = reinterpret_cast<v4i *>(blob);
    constexpr int U = 8;
    for (int32_t base = 0; base < n16; base += U * kWave) {
        v4i v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int32_t x = base + u * kWave + lane;
            v[u] = src[x < n16 ? x : n16 - 1];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int32_t x = base + u * kWave + lane;
            if (x < n16) dst[x] = v[u];
        }
    }
    int64_t *rg = reinterpret_cast<int64_t *>(blob + a.lds_member);
    rg[lane] = R.Jr;
    rg[kWave + lane] = R.Ar;
    rg[2 * kWave + lane] = R.Ur;
    if (RV == 2) {
        rg[3 * kWave + 3 + lane] = R.Jr2;
        rg[4 * kWave + 3 + lane] = R.Ar2;
    }
    if (lane == 0) {
        rg[3 * kWave] = R.s0;
        rg[3 * kWave + 1] = R.s1;
        rg[3 * kWave + 2] = R.s2;
    }
}
template <int RV>
__device__ inline void member_receive(const AnnealArgs &a, char *mine, const char *blob, Regs &R) {
    const int lane = lane_id();
    const int32_t n16 = a.lds_member >> 4;
    const v4i *src = reinterpret_cast<const v4i *>(blob);
    v4i *dst = reinterpret_cast<v4i *>(mine);
    const int64_t *rg = reinterpret_cast<const int64_t *>(blob + a.lds_member);
    R.Jr = rg[lane];
    R.Ar = rg[kWave + lane];
    R.Ur = rg[2 * kWave + lane];
    if (RV == 2) {
        R.Jr2 = rg[3 * kWave + 3 + lane];
        R.Ar2 = rg[4 * kWave + 3 + lane];
    }
    R.s0 = rg[3 * kWave];
    R.s1 = rg[3 * kWave + 1];
    R.s2 = rg[3 * kWave + 2];
    constexpr int U = 28;  // one batch covers a 28 KiB region
    for (int32_t base = 0; base < n16; base += U * kWave) {
        v4i v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int32_t x = base + u * kWave + lane;
            v[u] = src[x < n16 ? x : n16 - 1];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int32_t x = base + u * kWave + lane;
            if (x < n16) dst[x] = v[u];
        }
    }
    wsync();
}

// Stores and loads at device scope (every XCD): the store writes through to
// memory and the load reads from there, so data passed this way between
// workgroups needs no L2 writeback or invalidation around a barrier.
__device__ inline void st_dev(void *p, uint64_t v) {
    __hip_atomic_store(reinterpret_cast<uint64_t *>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline uint64_t ld_dev(const void *p) {
    return __hip_atomic_load(reinterpret_cast<const uint64_t *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Grid-wide barrier on a monotonic arrival counter; false if it timed out
// (then every workgroup stops).  Every thread of the workgroup takes part.
// FULL: release and acquire at agent scope (the XCD's L2 written back, then
// invalidated), so ordinary stores before it are visible to ordinary loads
// after it in every workgroup.  Otherwise only device-scope stores (st_dev)
// made before it are visible after it, to device-scope loads (ld_dev).
template <bool FULL>
__device__ inline bool grid_sync(unsigned *bar, unsigned target, int32_t *err, unsigned spin_limit, int32_t *s_ok) {
    if (!FULL) __builtin_amdgcn_s_waitcnt(0);  // this wave's st_dev stores have completed
    __syncthreads();
    if (threadIdx.x == 0) {
        if (FULL) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        __hip_atomic_fetch_add(bar, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        unsigned spins = 0;
        int32_t good = 1;
        while (__hip_atomic_load(bar, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
            __builtin_amdgcn_s_sleep(2);
            // (the error flag is polled every 32 spins: one load per spin)
            if ((++spins & 31) == 0 &&
                (spins > spin_limit || __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))) {
                __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                good = 0;
                break;
            }
        }
        if (FULL) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        *s_ok = good;
    }
    __syncthreads();
    return *s_ok != 0;
}

// Waits (one wave) until *p >= target, then acquires; false if it timed
// out or another wait or barrier failed (the error flag is set).
__device__ inline bool wave_wait_geq(const unsigned *p, unsigned target, int32_t *err, unsigned spin_limit) {
    unsigned spins = 0;
    for (;;) {
        unsigned v = 0;
        if (lane_id() == 0) v = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if ((unsigned)__builtin_amdgcn_readlane((int)v, 0) >= target) break;
        __builtin_amdgcn_s_sleep(2);
        if ((++spins & 31) == 0) {
            int32_t e = 0;
            if (lane_id() == 0) e = __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (spins > spin_limit || __builtin_amdgcn_readlane(e, 0)) {
                if (lane_id() == 0) __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                return false;
            }
        }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    return true;
}

// Systematic-resampling parent of a child: the first j with
// F_j P 2^32 >= rhs (F non-decreasing, the predicate holds at n - 1).  The
// search gallops from j0 in the direction the predicate asks, then bisects
// the bracket; near-uniform weights put the answer next to j0.
__device__ inline int32_t parent_search(const uint64_t *F, int32_t n, uint64_t P, unsigned __int128 rhs, int32_t j0) {
    auto ok = [&](int32_t j) { return (unsigned __int128)F[j] * P * ((uint64_t)1 << 32) >= rhs; };
    int32_t lo, hi;  // ok(hi) holds; ok(lo) fails (lo = -1: none known)
    if (ok(j0)) {
        hi = j0;
        lo = -1;
        for (int32_t step = 1; hi > 0; step <<= 1) {
            const int32_t c = hi - step < 0 ? 0 : hi - step;
            if (!ok(c)) {
                lo = c;
                break;
            }
            hi = c;
        }
    } else {
        lo = j0;
        hi = n - 1;
        for (int32_t step = 1; lo + step < n - 1; step <<= 1) {
            if (ok(lo + step)) {
                hi = lo + step;
                break;
            }
            lo += step;
        }
    }
    while (hi - lo > 1) {
        const int32_t md = lo + ((hi - lo) >> 1);
        if (ok(md)) hi = md;
        else lo = md;
    }
    return hi;
}

// Exclusive prefix over the workgroup of one value per thread (thread
// order); *total gets the sum.  Uses red[0 .. waves).
__device__ inline uint64_t block_excl_scan(uint64_t v, uint64_t *red, uint64_t *total) {
    const int lane = lane_id(), wv = wave_id(), nwv = blockDim.x / kWave;
    const uint64_t incl = wave_incl_scan_u(v);
    if (lane == kWave - 1) red[wv] = incl;
    __syncthreads();
    uint64_t base = 0, tot = 0;
    for (int w = 0; w < nwv; ++w) {
        base += w < wv ? red[w] : 0;
        tot += red[w];
    }
    __syncthreads();
    *total = tot;
    return base + incl - v;
}

}  // namespace



namespace {

template <int CTRL>
__device__ inline double fmin_step(double v) {
    const double o = __builtin_bit_cast(double, dpp64<CTRL>(__builtin_bit_cast(int64_t, v), __builtin_bit_cast(int64_t, v)));
    return o < v ? o : v;
}

// Minimum of doubles over the wave (no NaN); uniform.
__device__ inline double wave_min_f64(double v) {
    v = fmin_step<kDppXor1>(v);
    v = fmin_step<kDppXor2>(v);
    v = fmin_step<kDppHalfMirror>(v);
    v = fmin_step<kDppMirror>(v);
    double r = __builtin_bit_cast(double, (int64_t)readlane64((uint64_t)__builtin_bit_cast(int64_t, v), 0));
#pragma unroll
    for (int row = 1; row < 4; ++row) {
        const double o = __builtin_bit_cast(double, (int64_t)readlane64((uint64_t)__builtin_bit_cast(int64_t, v), 16 * row));
        r = o < r ? o : r;
    }
    return r;
}

}  // namespace

template <int PV, int DV, int GV, int LV>
__global__ void __launch_bounds__(kRunMaxWaves * kWave) k_anneal_chain_run(AnnealArgs a, RunArgs r) {
    extern __shared__ __align__(16) char smem[];
    __shared__ int64_t s_xs[3], s_k[kRunMaxWaves][4];
    __shared__ uint64_t s_red[kRunMaxWaves];
    __shared__ double s_dred[kRunMaxWaves];
    __shared__ int32_t s_win, s_ok;
    const Tables tb = load_tables<false>(a, smem);  // (never the CG layout)
    const int tid = threadIdx.x, nt = blockDim.x, lane = lane_id(), wv = wave_id(), nwv = nt / kWave;
    const int32_t pop = a.pop, N = a.N, K = a.K;
    const int gw = blockIdx.x * a.mpw + wv;  // this wave's slab
    const bool active = gw < pop;
    const int nb = gridDim.x;
    // level-end tables: in LDS, or (two row-shards per lane, whose member
    // regions leave no room) in this workgroup's slice of r.lend
    char *lend = GV == 2 ? r.lend + (int64_t)blockIdx.x * r.lend_stride : smem + r.o_lend;
    uint64_t *Fs = reinterpret_cast<uint64_t *>(lend);
    int32_t *par = reinterpret_cast<int32_t *>(Fs + pop);
    int32_t *flag = par + pop;    // has-child flags, then the slab -> next member map
    int32_t *freed = flag + pop;  // slabs of members without children, ascending member
    int32_t *slab = freed + pop;  // slab of each member
    int32_t *slabn = slab + pop;  // slab of each member after the hand-over
    for (int32_t j = tid; j < pop; j += nt) slab[j] = j;
    if (tid < 3) s_xs[tid] = r.xscore[tid];
    __syncthreads();
    Lds M{};
    SlabPtrs g{};
    Regs R{};
    int m = gw;
    if (active) {
        M = member_lds(a, smem, wv);
        g = slab_ptrs(a, a.slabs + (int64_t)gw * a.off.bytes);
        member_load<GV == 2 ? 2 : 1>(a, M, tb, g, R);
    }
    unsigned epoch = 0;
    const uint64_t P = (uint64_t)pop;
    const int32_t nW16 = a.RG * a.LP / 4;  // W of a slab in 16-byte units
    for (int n = 0; n < r.n_sweeps; ++n) {
        const int32_t level = r.offset + n;
        const double temp = r.temps[n];
        // ---- the level, then this workgroup's share of the level end
        int64_t k0 = LLONG_MAX, k1 = LLONG_MAX, k2 = LLONG_MAX, kj = LLONG_MAX;
        double emin = __builtin_inf();
        if (active) {
            const LevelOut lo = member_level<PV, DV, GV, LV, false>(
                a, M, tb, g.W, m, level, temp, s_xs[0], s_xs[1], s_xs[2],
                r.step_log ? r.step_log + ((int64_t)n * pop + m) * K : nullptr, a.results + (int64_t)m * kRes,
                r.trace ? r.trace + ((int64_t)n * pop + m) * 8 : nullptr, R);
            if (lane == 0) st_dev(r.energy + (int64_t)(n & 1) * pop + m, __builtin_bit_cast(uint64_t, lo.e));
            k0 = lo.b0;
            k1 = lo.b1;
            k2 = lo.b2;
            kj = m;
            emin = lo.e;
        }
        if (lane == 0) {
            s_k[wv][0] = k0; s_k[wv][1] = k1; s_k[wv][2] = k2; s_k[wv][3] = kj;
            s_dred[wv] = emin;
        }
        __syncthreads();
        if (tid == 0) {
            for (int w = 1; w < nwv; ++w) {
                if (lex_less(s_k[w][0], s_k[w][1], s_k[w][2], s_k[0][0], s_k[0][1], s_k[0][2]) ||
                    (s_k[w][0] == s_k[0][0] && s_k[w][1] == s_k[0][1] && s_k[w][2] == s_k[0][2] &&
                     s_k[w][3] < s_k[0][3]))
                    for (int f = 0; f < 4; ++f) s_k[0][f] = s_k[w][f];
                s_dred[0] = s_dred[w] < s_dred[0] ? s_dred[w] : s_dred[0];
            }
            for (int f = 0; f < 4; ++f)
                st_dev(r.wg_best + ((int64_t)(n & 1) * nb + blockIdx.x) * 4 + f, (uint64_t)s_k[0][f]);
            st_dev(r.wg_emin + (n & 1) * nb + blockIdx.x, __builtin_bit_cast(uint64_t, s_dred[0]));
        }
        // (the level's results cross workgroups by device-scope stores and
        // loads only: no L2 writeback here)
        if (!grid_sync<false>(r.bar, (unsigned)nb * ++epoch, r.err, r.spin_limit, &s_ok)) return;  // A

        // ---- every workgroup: incumbent and minimum energy from the workgroup summaries
        const double t_next = n + 1 < r.n_sweeps ? r.temps[n + 1] : r.t_after;
        const bool resample = t_next > 0.0;
        const int32_t per = (pop + nt - 1) / nt;
        const int32_t jlo = tid * per < pop ? tid * per : pop, jhi = jlo + per < pop ? jlo + per : pop;
        {
            k0 = k1 = k2 = kj = LLONG_MAX;
            emin = __builtin_inf();
            for (int b = tid; b < nb; b += nt) {
                const int64_t *wb = r.wg_best + ((int64_t)(n & 1) * nb + b) * 4;
                const int64_t v0 = (int64_t)ld_dev(wb), v1 = (int64_t)ld_dev(wb + 1), v2 = (int64_t)ld_dev(wb + 2),
                              vj = (int64_t)ld_dev(wb + 3);
                const double e = __builtin_bit_cast(double, ld_dev(r.wg_emin + (n & 1) * nb + b));
                if (lex_less(v0, v1, v2, k0, k1, k2) || (v0 == k0 && v1 == k1 && v2 == k2 && vj < kj)) {
                    k0 = v0; k1 = v1; k2 = v2; kj = vj;
                }
                emin = e < emin ? e : emin;
            }
            wave_lexmin(k0, k1, k2, kj);
            emin = wave_min_f64(emin);
            if (lane == 0) {
                s_k[wv][0] = k0; s_k[wv][1] = k1; s_k[wv][2] = k2; s_k[wv][3] = kj;
                s_dred[wv] = emin;
            }
            // the energies of this thread's members (used by the resampling weights)
            for (int32_t j = jlo; j < jhi; ++j) Fs[j] = ld_dev(r.energy + (int64_t)(n & 1) * pop + j);
            __syncthreads();
            if (tid == 0) {
                for (int w = 1; w < nwv; ++w) {
                    if (lex_less(s_k[w][0], s_k[w][1], s_k[w][2], s_k[0][0], s_k[0][1], s_k[0][2]) ||
                        (s_k[w][0] == s_k[0][0] && s_k[w][1] == s_k[0][1] && s_k[w][2] == s_k[0][2] &&
                         s_k[w][3] < s_k[0][3]))
                        for (int f = 0; f < 4; ++f) s_k[0][f] = s_k[w][f];
                    s_dred[0] = s_dred[w] < s_dred[0] ? s_dred[w] : s_dred[0];
                }
                const bool better = lex_less(s_k[0][0], s_k[0][1], s_k[0][2], s_xs[0], s_xs[1], s_xs[2]);
                s_win = better ? (int32_t)s_k[0][3] : -1;
                if (better) {
                    s_xs[0] = s_k[0][0];
                    s_xs[1] = s_k[0][1];
                    s_xs[2] = s_k[0][2];
                }
            }
            __syncthreads();
        }
        // A level that moved the incumbent reads rows that members wrote
        // with ordinary stores (the winner's trajectory best here, the
        // parents' W rows below): a full barrier first.
        const bool sync_b = s_win >= 0;
        if (sync_b && !grid_sync<true>(r.bar, (unsigned)nb * ++epoch, r.err, r.spin_limit, &s_ok)) return;
        if (sync_b) {
            // x* := the winner's trajectory best, one slice per workgroup
            const int32_t sl = (N + nb - 1) / nb, x0 = blockIdx.x * sl, x1 = x0 + sl < N ? x0 + sl : N;
            const int32_t *src = a.best + (int64_t)s_win * N;
            for (int32_t x = x0 + tid; x < x1; x += nt) r.xstar[x] = src[x];
            if (blockIdx.x == 0 && tid < 3) r.xscore[tid] = s_xs[tid];
        }
        // ---- systematic resampling with quantised Boltzmann weights
        if (resample) {
            emin = s_dred[0];
            const double den = fabs(emin) > 1.0 ? fabs(emin) : 1.0;
            const double cfac = (1.0 / t_next) - (1.0 / temp);
            uint64_t local = 0;
            for (int32_t j = jlo; j < jhi; ++j) {
                const double en = (__builtin_bit_cast(double, Fs[j]) - emin) / den;
                const uint64_t w = (uint64_t)floor(__builtin_ldexp(exp_det(-(cfac * en)), 40));
                Fs[j] = w;
                local += w;
            }
            uint64_t total = 0;
            uint64_t run = block_excl_scan(local, s_red, &total);
            for (int32_t j = jlo; j < jhi; ++j) {
                run += Fs[j];
                Fs[j] = run;
            }
            __syncthreads();
            const uint64_t V = r.vwords[n];
            // children of this thread: [jlo, jhi); parents are non-decreasing
            int32_t pj = jlo < pop ? jlo : pop - 1;
            for (int32_t mm = jlo; mm < jhi; ++mm) {
                const unsigned __int128 rhs = (unsigned __int128)total * (V + ((uint64_t)mm << 32));
                pj = parent_search(Fs, pop, P, rhs, pj);
                par[mm] = pj;
            }
            for (int32_t mm = tid; mm < pop; mm += nt) flag[mm] = 0;
        } else {
            for (int32_t mm = tid; mm < pop; mm += nt) par[mm] = mm;
        }
        __syncthreads();
        if (r.parents_out) {
            const int32_t sl = (pop + nb - 1) / nb, p0 = blockIdx.x * sl, p1 = p0 + sl < pop ? p0 + sl : pop;
            for (int32_t mm = p0 + tid; mm < p1; mm += nt)
                r.parents_out[(int64_t)n * pop + mm] = resample ? par[mm] : -1;
        }
        // ---- slab hand-over
        // A level that moved the incumbent ends with grid barrier B (x* is
        // copied from a member's trajectory-best row, which the next level
        // may overwrite).  Otherwise the hand-over is point to point: a
        // publisher releases its image with a flag; each receiver waits for
        // that flag, copies the image and the parent's W into its own slab
        // and counts itself in; the publisher, whose first child keeps the
        // parent's slab, waits for that count before its next level changes
        // W.  s_win is the same in every workgroup, so all of them take the
        // same path.
        const unsigned token = (unsigned)n + 1;  // (flags are zero at launch)
        int32_t m_next = m, src_slab = -1, n_recv = 0;
        bool publish = false;
        if (resample) {
            // bit 0: the member has a child; bit 1: a second one
            for (int32_t mm = tid; mm < pop; mm += nt)
                atomicOr(&flag[par[mm]], (mm > 0 && par[mm - 1] == par[mm]) ? 3 : 1);
            __syncthreads();
            // the current member publishes its state when it has a second child
            publish = active && (flag[m] & 2) != 0;
            int32_t n_dead = 0, n_dup = 0;
            for (int32_t j = jlo; j < jhi; ++j) {
                n_dead += (flag[j] & 1) == 0;
                n_dup += (j > 0 && par[j] == par[j - 1]);
            }
            uint64_t tdead = 0, tdup = 0;
            int32_t rdead = (int32_t)block_excl_scan((uint64_t)n_dead, s_red, &tdead);
            int32_t rdup = (int32_t)block_excl_scan((uint64_t)n_dup, s_red, &tdup);
            for (int32_t j = jlo; j < jhi; ++j)
                if ((flag[j] & 1) == 0) freed[rdead++] = slab[j];
            __syncthreads();
            int32_t *dups = reinterpret_cast<int32_t *>(Fs);  // further children, ascending
            for (int32_t mm = jlo; mm < jhi; ++mm) {
                const int32_t pp = par[mm];
                if (mm == 0 || pp != par[mm - 1]) {
                    slabn[mm] = slab[pp];
                } else {
                    dups[rdup] = mm;
                    slabn[mm] = freed[rdup++];
                }
            }
            __syncthreads();
            for (int32_t mm = tid; mm < pop; mm += nt) flag[slabn[mm]] = mm;  // slab -> next member
            __syncthreads();
            if (active) {
                m_next = flag[gw];
                const int32_t pn = par[m_next];
                if (m_next > 0 && par[m_next - 1] == pn) src_slab = slab[pn];
                if (publish) {  // the further children of this member
                    int32_t c = m_next + 1;
                    while (c < pop && par[c] == pn) ++c;
                    n_recv = c - m_next - 1;
                }
            }
            // Every further child gets its parent's W in its own slab; with
            // barrier B the copies are split evenly over all workgroups.
            if (sync_b) {
                // units <= pop * nW16 < 2^31: nW16 <= 128 * 32 * 16 / 4 and the
                // level-end tables in LDS hold pop below 6000
                const int32_t *dups = reinterpret_cast<const int32_t *>(Fs);
                const int32_t units = (int32_t)tdup * nW16;
                const int32_t share = (units + nb - 1) / nb;
                const int32_t u0 = blockIdx.x * share, u1 = u0 + share < units ? u0 + share : units;
                constexpr int U = 4;
                for (int32_t base = u0; base < u1; base += U * nt) {
                    // every slot loads (clamped to the last unit), so all U
                    // loads are in flight before the first store
                    v4i v[U];
                    int64_t dsto[U];
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        const int32_t x = base + u * nt + tid < u1 ? base + u * nt + tid : u1 - 1;
                        const int32_t ci = (int32_t)((uint32_t)x / (uint32_t)nW16);
                        const int32_t off = x - ci * nW16;
                        const int32_t c = dups[ci];
                        v[u] = reinterpret_cast<const v4i *>(a.slabs + (int64_t)slab[par[c]] * a.off.bytes + a.off.W)[off];
                        dsto[u] = (int64_t)slabn[c] * a.off.bytes + a.off.W + (int64_t)off * 16;
                    }
#pragma unroll
                    for (int u = 0; u < U; ++u)
                        if (base + u * nt + tid < u1) *reinterpret_cast<v4i *>(a.slabs + dsto[u]) = v[u];
                }
            }
            // and the rest of its state from the parent's own slab
            if (publish) {
                member_publish<GV == 2 ? 2 : 1>(a, smem + a.lds_shared + (int64_t)wv * a.lds_member, r.blobs + (int64_t)gw * r.blob_bytes, R);
                if (!sync_b) {
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
                    if (lane == 0) __hip_atomic_store(r.pub + gw, token, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
            }
        }
        if (sync_b && !grid_sync<true>(r.bar, (unsigned)nb * ++epoch, r.err, r.spin_limit, &s_ok)) return;  // B
        if (resample) {
            for (int32_t mm = tid; mm < pop; mm += nt) slab[mm] = slabn[mm];
            __syncthreads();
            char *mine = smem + a.lds_shared + (int64_t)wv * a.lds_member;
            if (active && src_slab >= 0 && (sync_b || wave_wait_geq(r.pub + src_slab, token, r.err, r.spin_limit))) {
                member_receive<GV == 2 ? 2 : 1>(a, mine, r.blobs + (int64_t)src_slab * r.blob_bytes, R);
                if (!sync_b) {
                    wave_copy16(a.slabs + (int64_t)src_slab * a.off.bytes + a.off.W,
                                a.slabs + (int64_t)gw * a.off.bytes + a.off.W, nW16);
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
                    if (lane == 0) __hip_atomic_fetch_add(r.got + src_slab, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
            }
            if (!sync_b && publish && wave_wait_geq(r.got + gw, (unsigned)n_recv, r.err, r.spin_limit) && lane == 0)
                __hip_atomic_store(r.got + gw, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (!sync_b) {
                // A wait that gave up has set the error flag: the whole
                // workgroup leaves before a wave starts the next level on a
                // state that was not received, or writes W rows that a
                // receiver may still be copying.
                __syncthreads();
                if (tid == 0) s_ok = __hip_atomic_load(r.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0;
                __syncthreads();
                if (!s_ok) return;
            }
        }
        m = m_next;
    }
    if (active) member_store<GV == 2 ? 2 : 1>(a, M, g, R);
    if (blockIdx.x == 0)
        for (int32_t mm = tid; mm < pop; mm += nt) r.slab_of_out[mm] = slab[mm];
}

// Resampling offset words (Alg. 3 reweighting step): V of a level is the
// high half of the first word of the tag-2 Philox block with counter
// (0, level, 2^32 - 1, 2); one thread per level.
__global__ void __launch_bounds__(256) k_resample_words(uint64_t seed, int32_t offset, int32_t n, uint32_t *v) {
    const int32_t x = blockIdx.x * blockDim.x + threadIdx.x;
    if (x >= n) return;
    const U64x4 blk = philox4x64_10(0, (uint64_t)(uint32_t)(offset + x), 0xFFFFFFFFull, 2, seed, 0);
    v[x] = (uint32_t)(blk.v[0] >> 32);
}

int launch_resample_words(uint64_t seed, int32_t offset, int32_t n, uint32_t *v, hipStream_t stream) {
    if (n <= 0) return ROUTEPACK_OK;
    hipLaunchKernelGGL(k_resample_words, dim3((n + 255) / 256), dim3(256), 0, stream, seed, offset, n, v);
    return hipGetLastError() == hipSuccess ? ROUTEPACK_OK : ROUTEPACK_E_DEVICE;
}

// Rows of L x P int32 from layer-major [L][P] to chunk-major [P/4][L][4],
// one row per workgroup (in place when src == dst).
__global__ void __launch_bounds__(256) k_rows_to_chunks(const int32_t *src, int32_t *dst, int64_t n_rows,
                                                      int64_t row_stride, int64_t rows_per_group,
                                                      int64_t group_stride, int32_t L, int32_t P) {
    __shared__ int32_t row[4096];  // L * P <= 64 * 64
    const int64_t rr = blockIdx.x;
    if (rr >= n_rows) return;
    const int64_t off = (rr / rows_per_group) * group_stride + (rr % rows_per_group) * row_stride;
    const int32_t LP = L * P;
    for (int32_t e = threadIdx.x; e < LP; e += blockDim.x) row[e] = src[off + e];
    __syncthreads();
    for (int32_t e = threadIdx.x; e < LP; e += blockDim.x) {
        const int32_t l = e / P, p = e - l * P;
        dst[off + ((p >> 2) * L + l) * 4 + (p & 3)] = row[e];
    }
}

int chain_prepare(AnnealArgs &a, int32_t *qt, hipStream_t stream) {
    if (a.L * a.P > 4096 || (a.P & 3) != 0) return ROUTEPACK_E_UNSUPPORTED;
    if (a.LP > 0) {
        hipLaunchKernelGGL(k_rows_to_chunks, dim3((unsigned)a.N), dim3(256), 0, stream, a.q, qt, (int64_t)a.N,
                           (int64_t)a.LP, (int64_t)1, (int64_t)a.LP, a.L, a.P);
        int32_t *w = reinterpret_cast<int32_t *>(a.slabs + a.off.W);
        const int64_t rows = (int64_t)a.pop * a.RG;
        hipLaunchKernelGGL(k_rows_to_chunks, dim3((unsigned)rows), dim3(256), 0, stream, w, w, rows, (int64_t)a.LP,
                           (int64_t)a.RG, a.off.bytes / (int64_t)sizeof(int32_t), a.L, a.P);
        if (hipGetLastError() != hipSuccess) return ROUTEPACK_E_DEVICE;
    }
    a.qt = qt;
    return ROUTEPACK_OK;
}

// Launch shape of the chain kernel; false when the problem is outside its
// shape (the caller then uses the flat wave kernel).
bool chain_plan(AnnealArgs &a, int32_t n_cu, int32_t max_count, int32_t *pv_out, int32_t *dv_out) {
    const int32_t P = a.P;
    if (!(P == 4 || P == 8 || P == 16 || P == 32 || P == 64)) return false;
    // (L >= 1: each move loads its rows with a layer on every lane of a half;
    // 33 to 64 layers take two layers per lane, compiled for P >= 16; up to
    // 16 slots per row-shard, or 32 with 64 ranks)
    if (a.L < 1 || a.L > 64 || (a.L > 32 && P < 16) || a.RG > 2 * kWave || max_count > (P == 64 ? 32 : 16) ||
        a.N > 65535 || a.B + 1 > 65535 || a.C > 2147483647LL)
        return false;
    // (32 or 64 ranks with two row-shards per lane are not compiled)
    if (P >= 32 && a.RG > kWave) return false;
    a.lv = a.L > 32 ? 2 : 1;
    a.rv = a.RG > kWave ? 2 : 1;  // row-shards per lane
    // (64 ranks are compiled with 32 slot lanes and the HBM layout only)
    const int32_t dv = P == 64 ? 32 : (max_count <= 8 ? 8 : 16);
    a.dv = dv;
    a.ginv = (uint32_t)((((uint64_t)1 << 32) + (uint64_t)a.G - 1) / (uint64_t)a.G);
    a.dinv = (uint32_t)((((uint64_t)1 << 32) + (uint64_t)a.D - 1) / (uint64_t)a.D);
    a.dshift = -1;
    for (int32_t sh = 0; sh < 16; ++sh)
        if ((1 << sh) == a.D) a.dshift = sh;
    auto up16 = [](int64_t x) { return (x + 15) & ~(int64_t)15; };
    auto up8e = [](int64_t n) { return ((n + 7) & ~(int64_t)7) + 16; };  // elements, padded for 16-byte steps
    // 64 ranks: the pool and Q stay in the slab and the cost prefixes in a
    // per-member HBM array (a member's LDS is then its start offsets, cell
    // loads and roulette prefixes, about 13 KB for the largest window)
    const bool hq = P == 64;
    a.hq = hq ? 1 : 0;
    a.cp_stride = hq ? (int32_t)((((int64_t)a.RG * (dv + 1) + a.RG) + 3) & ~(int64_t)3) : 0;
    // LDS of one member and of the workgroup's shared tables; with cg the
    // cell array stays in the slab and the lengths are read from HBM.
    auto layout = [&](bool cg, int64_t *shared_out) -> int64_t {
        int64_t o = 0;
        a.o_cell = (int32_t)o; o = up16(o + (cg ? 0 : 2 * (int64_t)a.N));
        a.o_pool = (int32_t)o; o = up16(o + (hq && cg ? 0 : 2 * up8e(a.N)));
        a.o_start = (int32_t)o; o = up16(o + 2 * up8e((int64_t)a.B + 1));
        a.o_T = (int32_t)o; o = up16(o + 4 * (int64_t)a.B);
        a.o_Q = (int32_t)o; o = up16(o + (hq ? 0 : 8 * (int64_t)a.B));
        a.o_acost = (int32_t)o; o = up16(o + (hq ? 0 : 8 * ((int64_t)a.RG * (dv + 1) + a.RG)));  // cost prefixes and totals
        a.o_Jpre = (int32_t)o; o = up16(o + 8 * 144 * (int64_t)a.rv);  // J_pre, V_pre and their pivots
        a.o_Jpiv = a.o_Jpre + 8 * 128 * a.rv;
        int64_t tab = up16(4 * ((int64_t)a.G * a.D + 2 * a.G + a.D));
        a.o_hcnt = (int32_t)tab; tab = up16(tab + 4 * (int64_t)a.RG);
        a.o_hcell = (int32_t)tab; tab = up16(tab + (hq && a.G == 1 ? 0 : 4 * (int64_t)a.RG * dv));
        a.o_tshared = (int32_t)tab;
        *shared_out = up16(tab + (cg ? 0 : 4 * (int64_t)a.N));
        return o;
    };
    const int64_t lim = 160 * 1024;
    int64_t want = ((int64_t)a.pop + n_cu - 1) / n_cu;
    want = want < 1 ? 1 : (want > kRunMaxWaves ? kRunMaxWaves : want);
    int64_t shared = 0, member = layout(false, &shared);
    int64_t cap = shared + member <= lim ? (lim - shared) / member : 0;
    a.cg = 0;
    // ROUTEPACK_CHAIN_LAYOUT=hbm asks for the HBM layout (P = 32), =lds forbids it
    const char *lay = getenv("ROUTEPACK_CHAIN_LAYOUT");
    const bool force_hbm = lay && strcmp(lay, "hbm") == 0, no_hbm = lay && strcmp(lay, "lds") == 0;
    if (force_hbm && P < 32) return false;
    if (P == 64 && no_hbm) return false;
    if (((cap < want && !no_hbm) || force_hbm || P == 64) && P >= 32) {
        // the population cannot be resident at once (or 64 ranks): more
        // members per CU with the cell array and the lengths in HBM
        // (compiled for P = 32 and 64)
        int64_t shared_g = 0;
        const int64_t member_g = layout(true, &shared_g);
        const int64_t cap_g = shared_g + member_g <= lim ? (lim - shared_g) / member_g : 0;
        if (cap_g > cap || ((force_hbm || P == 64) && cap_g >= 1)) {
            a.cg = 1;
            shared = shared_g;
            member = member_g;
            cap = cap_g;
        } else {
            layout(false, &shared);
        }
    }
    if (cap < 1 || (P == 64 && !a.cg)) return false;
    a.mpw = (int32_t)(want < cap ? want : cap);
    a.lds_shared = (int32_t)shared;
    a.lds_member = (int32_t)member;
    *pv_out = P;
    *dv_out = dv;
    return true;
}

template <int PV, int DV, int GV, int LV, bool CG>
static int chain_launch_t(const AnnealArgs &a, hipStream_t stream) {
    const size_t lds = (size_t)a.lds_shared + (size_t)a.mpw * a.lds_member;
    if (hipFuncSetAttribute((const void *)k_anneal_chain<PV, DV, GV, LV, CG>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
        return ROUTEPACK_E_DEVICE;
    const unsigned grid = (unsigned)((a.pop + a.mpw - 1) / a.mpw);
    hipLaunchKernelGGL((k_anneal_chain<PV, DV, GV, LV, CG>), dim3(grid), dim3(kWave * a.mpw), lds, stream, a);
    return hipGetLastError() == hipSuccess ? ROUTEPACK_OK : ROUTEPACK_E_DEVICE;
}

// Level-end tables of the whole-schedule kernel (after the member regions,
// or in HBM for the two-per-lane variant).
int64_t run_lend_bytes(int32_t pop) { return (28 * (int64_t)pop + 255) & ~(int64_t)255; }

template <int PV, int DV, int GV, int LV>
static int chain_run_t(const AnnealArgs &a, const RunArgs &r0, int32_t n_cu, bool launch, hipStream_t stream) {
    RunArgs r = r0;
    if (a.mpw > kRunMaxWaves) return ROUTEPACK_E_UNSUPPORTED;
    const int64_t o_lend = ((int64_t)a.lds_shared + (int64_t)a.mpw * a.lds_member + 15) & ~(int64_t)15;
    const int64_t lds = o_lend + (GV == 2 ? 0 : run_lend_bytes(a.pop));
    if (GV == 2 && launch && (!r.lend || r.lend_stride < run_lend_bytes(a.pop))) return ROUTEPACK_E_INTERNAL;
    // static LDS of the kernel is below 1 KiB
    if (lds + 1024 > 160 * 1024) return ROUTEPACK_E_UNSUPPORTED;
    r.o_lend = (int32_t)o_lend;
    const void *fn = (const void *)k_anneal_chain_run<PV, DV, GV, LV>;
    if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
        return ROUTEPACK_E_DEVICE;
    const int grid = (a.pop + a.mpw - 1) / a.mpw, block = kWave * a.mpw;
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, block, (size_t)lds) != hipSuccess)
        return ROUTEPACK_E_DEVICE;
    if ((int64_t)per_cu * n_cu < grid) return ROUTEPACK_E_UNSUPPORTED;  // not all resident
    if (!launch) return ROUTEPACK_OK;
    AnnealArgs aa = a;
    void *args[] = {&aa, &r};
    if (hipLaunchCooperativeKernel(fn, dim3(grid), dim3(block), args, (unsigned)lds, stream) != hipSuccess)
        return ROUTEPACK_E_DEVICE;
    return hipGetLastError() == hipSuccess ? ROUTEPACK_OK : ROUTEPACK_E_DEVICE;
}

// The variant of the chain kernels for this problem: 2 with more than 64
// row-shards, else 1 for the common shape and 0 for the general one.
static int chain_variant(const AnnealArgs &a, bool step_log) {
    if (a.rv == 2) return 2;
    return a.G == 1 && a.dshift >= 0 && a.S == 1 && a.sum32 && a.scale_pow2 && !step_log ? 1 : 0;
}

template <int PV, int DV, int LV>
static int chain_run_v(int v, const AnnealArgs &a, const RunArgs &r, int32_t n_cu, bool launch, hipStream_t stream) {
    if (v == 2) {
        if constexpr (PV == 32) return ROUTEPACK_E_UNSUPPORTED;  // (excluded by chain_plan)
        else return chain_run_t<PV, DV, 2, LV>(a, r, n_cu, launch, stream);
    }
    if (v == 1) return chain_run_t<PV, DV, 1, LV>(a, r, n_cu, launch, stream);
    return chain_run_t<PV, DV, 0, LV>(a, r, n_cu, launch, stream);
}

template <int DV>
static int chain_run_d(int v, const AnnealArgs &a, const RunArgs &r, int32_t pv, int32_t n_cu, bool launch,
                       hipStream_t stream) {
    if (a.lv == 2) {
        switch (pv) {
            case 16: return chain_run_v<16, DV, 2>(v, a, r, n_cu, launch, stream);
            case 32: return chain_run_v<32, DV, 2>(v, a, r, n_cu, launch, stream);
        }
        return ROUTEPACK_E_UNSUPPORTED;
    }
    switch (pv) {
        case 4: return chain_run_v<4, DV, 1>(v, a, r, n_cu, launch, stream);
        case 8: return chain_run_v<8, DV, 1>(v, a, r, n_cu, launch, stream);
        case 16: return chain_run_v<16, DV, 1>(v, a, r, n_cu, launch, stream);
        case 32: return chain_run_v<32, DV, 1>(v, a, r, n_cu, launch, stream);
    }
    return ROUTEPACK_E_UNSUPPORTED;
}

// Checks (launch = false) or launches (launch = true) the whole-schedule
// kernel; ROUTEPACK_E_UNSUPPORTED when its workgroups cannot all be resident.
int chain_run(const AnnealArgs &a, const RunArgs &r, int32_t pv, int32_t dv, int32_t n_cu, bool launch,
              hipStream_t stream) {
    // (only the per-level kernel is compiled for the HBM layout and 64 ranks)
    if (a.cg || dv == 32) return ROUTEPACK_E_UNSUPPORTED;
    const int v = chain_variant(a, r.step_log != nullptr);
    return dv == 8 ? chain_run_d<8>(v, a, r, pv, n_cu, launch, stream)
                   : chain_run_d<16>(v, a, r, pv, n_cu, launch, stream);
}

template <int PV, int DV, int LV>
static int chain_launch_v(int v, const AnnealArgs &a, hipStream_t stream) {
    if constexpr (PV >= 32) {
        if (v == 2) return ROUTEPACK_E_UNSUPPORTED;  // (excluded by chain_plan)
        if (a.cg) return v == 1 ? chain_launch_t<PV, DV, 1, LV, true>(a, stream)
                                : chain_launch_t<PV, DV, 0, LV, true>(a, stream);
    } else {
        if (a.cg) return ROUTEPACK_E_UNSUPPORTED;  // (chain_plan takes it for P = 32 and 64 only)
        if (v == 2) return chain_launch_t<PV, DV, 2, LV, false>(a, stream);
    }
    if constexpr (PV == 64) {
        return ROUTEPACK_E_UNSUPPORTED;  // (64 ranks: the HBM layout only)
    } else {
        if (v == 1) return chain_launch_t<PV, DV, 1, LV, false>(a, stream);
        return chain_launch_t<PV, DV, 0, LV, false>(a, stream);
    }
}

template <int DV>
static int chain_launch_d(int v, const AnnealArgs &a, int32_t pv, hipStream_t stream) {
    if (a.lv == 2) {
        switch (pv) {
            case 16: return chain_launch_v<16, DV, 2>(v, a, stream);
            case 32: return chain_launch_v<32, DV, 2>(v, a, stream);
        }
        return ROUTEPACK_E_UNSUPPORTED;
    }
    switch (pv) {
        case 4: return chain_launch_v<4, DV, 1>(v, a, stream);
        case 8: return chain_launch_v<8, DV, 1>(v, a, stream);
        case 16: return chain_launch_v<16, DV, 1>(v, a, stream);
        case 32: return chain_launch_v<32, DV, 1>(v, a, stream);
    }
    return ROUTEPACK_E_UNSUPPORTED;
}

int launch_anneal_chain(const AnnealArgs &a, int32_t pv, int32_t dv, hipStream_t stream) {
    const int v = chain_variant(a, a.step_log != nullptr);
    if (dv == 32) {  // (64 ranks only)
        if (pv != 64) return ROUTEPACK_E_UNSUPPORTED;
        return a.lv == 2 ? chain_launch_v<64, 32, 2>(v, a, stream) : chain_launch_v<64, 32, 1>(v, a, stream);
    }
    return dv == 8 ? chain_launch_d<8>(v, a, pv, stream) : chain_launch_d<16>(v, a, pv, stream);
}

}  // namespace rp
