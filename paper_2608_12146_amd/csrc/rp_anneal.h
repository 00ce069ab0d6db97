// Shared declarations of the annealing kernels (one-workgroup-per-member
// fallback in rp_anneal.hip, one-wave-per-member kernel in
// rp_anneal_wave.hip): member slab layout, kernel arguments and wave-level
// helpers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rp_device.h"
#include "rp_internal.h"

namespace rp {

constexpr int kThreads = 256;
constexpr int kMaxEPT = 16;   // W entries per thread: L*P <= 4096
constexpr int kMaxJPL = 8;    // row-shards per lane: R*G <= 512
constexpr int kMaxStages = 4;
constexpr int kRes = 10;      // per-member result words

struct SlabOffsets {
    int64_t cell, pool, start, T, Q, W, J, A, bytes;
};

struct AnnealArgs {
    const int32_t *t, *q;
    int32_t N, L, P, D, G, R, S, F, K;
    int32_t LP, RG, B, nx, pshift;
    int64_t C;
    double scale, temp;
    int64_t alpha[kMaxStages], beta[kMaxStages];
    const int32_t *slots, *count, *slot_shard;
    char *src, *dst;
    SlabOffsets off;
    const int32_t *parent;  // [pop] or null (identity)
    int32_t *best;          // [pop][N]
    int64_t *results;       // [pop][kRes]
    uint8_t *step_log;      // [pop][K] or null
    uint64_t seed;
    int32_t level;
    uint32_t p_guide, rho;
    // one-wave-per-member kernel
    char *slabs;              // single slab buffer, members updated in place
    const int32_t *slab_of;   // [pop] slab of each member
    const int64_t *xscore;    // [3] incumbent score at the level start
    int32_t pop, mpw;         // population, members per workgroup
    int32_t lds_shared, lds_member;
    int32_t o_cell, o_pool, o_start, o_T, o_Q, o_acost, o_Jpre;
    int32_t o_Jpiv, o_tshared;  // chain kernel: J pivots (per member), lengths table (shared)
    uint32_t ginv, dinv;        // chain kernel: ceil(2^32 / G), ceil(2^32 / D) (unused when G, D == 1)
    int32_t dshift;             // chain kernel: log2 D when D is a power of two, else -1
    int32_t rv;                 // chain kernel: row-shards per lane (1 up to 64 row-shards, 2 up to 128)
    int32_t lv;                 // chain kernel: layers per lane (1 up to 32 layers, 2 up to 64)
    int32_t cg;                 // chain kernel: the cell array and the lengths stay in HBM, not LDS
    int32_t hq;                 // chain kernel (64 ranks): Q in the slab and the cost prefixes in gcp, not LDS
    int64_t *gcp;               // [pop][cp_stride] cost prefixes and totals of each member (hq)
    int32_t cp_stride;
    int32_t dv, o_hcnt, o_hcell;  // chain kernel: cost-prefix stride; row-shard slot tables (shared)
    int32_t scale_pow2;         // 2^F C is a power of two
    double inv_scale;           // 1 / (2^F C) when it is
    unsigned long long *phase_cycles;  // [pop][8] with RP_PHASE_TIMERS builds, else unused
    const int32_t *qzero;       // [L * P] zeros (chain kernels: the q row of "no sample")
    const int32_t *qt;          // chain kernels: q rows in chunk-major order [N][P/4][L][4]
    int32_t sum32;              // L * (W entry bound) < 2^31: per-row layer sums fit int32
};

// Wave kernel plan and launchers (rp_anneal_wave.hip).
bool wave_plan(AnnealArgs &a, int32_t n_cu, int32_t *mpw_out, bool *tlds_out);
int launch_anneal_wave(const AnnealArgs &a, bool tlds, hipStream_t stream);
// Arguments of the whole-schedule chain kernel (rp_anneal_chain.hip).
struct RunArgs {
    const double *temps;   // [n_sweeps] (device)
    int32_t n_sweeps, offset;
    double t_after;        // temperature after the last level; <= 0: no resampling after it
    int64_t *trace;        // [n_sweeps][pop][8] or null
    int32_t *parents_out;  // [n_sweeps][pop] or null
    uint8_t *step_log;     // [n_sweeps][pop][K] or null
    int32_t *xstar;        // [N]
    int64_t *xscore;       // [3]
    unsigned *bar;         // grid barrier arrivals (zero at launch)
    int32_t *err;          // set when a grid barrier times out
    int32_t *slab_of_out;  // [pop] slab of each member after the run
    double *energy;        // [2][pop] terminal energy of each member (by level parity)
    int64_t *wg_best;      // [2][workgroups][4] lexicographic-min trajectory best and its member
    double *wg_emin;       // [2][workgroups] minimum terminal energy
    int32_t o_lend;        // LDS offset of the level-end tables
    char *lend;            // [workgroups][lend_stride] level-end tables in HBM (two row-shards per lane)
    int64_t lend_stride;
    char *blobs;           // [pop][blob_bytes]: a published member's LDS image and registers, per slab
    int64_t blob_bytes;
    unsigned *pub;         // [pop] per slab: the last level whose image it published (zero at launch)
    unsigned *got;         // [pop] per slab: receivers that have copied its image (zero at launch)
    unsigned spin_limit;   // polls before a barrier or hand-over wait gives up (sets err)
    const uint32_t *vwords;  // [n_sweeps] resampling offset word V of each level (tag-2 Philox block)
};

// V of levels offset .. offset + n - 1 into v (the run kernel reads them at
// each level end instead of drawing the Philox block there).
int launch_resample_words(uint64_t seed, int32_t offset, int32_t n, uint32_t *v, hipStream_t stream);

// Bytes of the whole-schedule kernel's level-end tables for a population.
int64_t run_lend_bytes(int32_t pop);

// Bytes of one hand-over image: the member's LDS region, then J, A and U of
// every lane, the score, and J and A of the lanes' second row-shards.
inline int64_t run_blob_bytes(int32_t lds_member) { return ((int64_t)lds_member + 8 * (5 * 64 + 3) + 255) & ~(int64_t)255; }

// Chain kernels: rows of L x P int32 are kept chunk-major, [P/4][L][4], so a
// 16-byte access of every lane of a half-wave (lane = layer) is contiguous.
// Rewrites the W rows of every slab in place and writes qt (N rows).
int chain_prepare(AnnealArgs &a, int32_t *qt, hipStream_t stream);
// Chain kernel plan and launchers (rp_anneal_chain.hip).
bool chain_plan(AnnealArgs &a, int32_t n_cu, int32_t max_count, int32_t *pv_out, int32_t *dv_out);
int launch_anneal_chain(const AnnealArgs &a, int32_t pv, int32_t dv, hipStream_t stream);
int chain_run(const AnnealArgs &a, const RunArgs &r, int32_t pv, int32_t dv, int32_t n_cu, bool launch,
              hipStream_t stream);
int launch_copy_slabs(char *slabs, int64_t bytes, const int32_t *src, const int32_t *dst,
                      const int32_t *n_copies, int32_t pop, hipStream_t stream);

template <class T>
__device__ __host__ inline T *at(char *base, int64_t off) {
    return reinterpret_cast<T *>(base + off);
}


// Roulette over non-negative weights held one per lane (index = base + lane,
// n indices in total, over JPL register chunks): pick = bounded(word, total),
// result = the first index whose inclusive prefix exceeds pick; all-zero
// weights fall back to a uniform index.
template <int JPL>
__device__ inline int roulette_chunks(const int64_t (&w)[JPL], int n, uint64_t word,
                                      int64_t total) {
    if (total == 0) return (int)bounded(word, (uint64_t)n);
    const uint64_t pick = bounded(word, (uint64_t)total);
    const int lane = lane_id();
    int64_t carry = 0;
#pragma unroll
    for (int x = 0; x < JPL; ++x) {
        if (x * kWave < n) {
            const int h = x * kWave + lane;
            const int64_t v = h < n ? w[x] : 0;
            const int64_t incl = wave_incl_scan(v) + carry;
            const uint64_t mask = __ballot(h < n && (uint64_t)incl > pick);
            if (mask) return x * kWave + first_lane(mask);
            carry = (int64_t)readlane64((uint64_t)incl, kWave - 1);
        }
    }
    return n - 1;
}

__device__ inline int32_t clampi(int32_t v, int32_t lo, int32_t hi) {
    return v < lo ? lo : (v > hi ? hi : v);
}

// #{x in pool[lo, hi) : x < v and x != skip}, uniform over the wave.
__device__ inline int32_t seg_count_less(const int32_t *pool, int32_t lo, int32_t hi, int32_t v,
                                         int32_t skip, int32_t limit) {
    int32_t cnt = 0;
    const int lane = lane_id();
    lo = lo < 0 ? 0 : lo;
    hi = hi > limit ? limit : hi;
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

// Remove the element at `from`, insert v at `to`, shifting the elements in
// between by one; every thread of the block takes part (uniform arguments).
__device__ inline void pool_move(int32_t *pool, int32_t from, int32_t to, int32_t v) {
    const int tid = threadIdx.x;
    if (from < to) {
        for (int32_t base = from; base < to; base += kThreads) {
            const int32_t x = base + tid;
            int32_t val = 0;
            if (x < to) val = pool[x + 1];
            __syncthreads();
            if (x < to) pool[x] = val;
            __syncthreads();
        }
    } else if (from > to) {
        for (int32_t top = from; top > to; top -= kThreads) {
            const int32_t x = top - tid;
            int32_t val = 0;
            if (x > to) val = pool[x - 1];
            __syncthreads();
            if (x > to) pool[x] = val;
            __syncthreads();
        }
    }
    if (tid == 0) pool[to] = v;
    __syncthreads();
}

// Attention part A(r, g) = sum_s max_{x < count[g]} cost_s(cell x of the
// row-shard), with up to two cells' statistics replaced.  Uniform over the
// wave; requires count[g] <= 64.
__device__ inline int64_t attention_rs(const AnnealArgs &a, const int64_t *T, const int64_t *Q,
                                       int32_t r, int32_t g, int32_t c1, int64_t T1, int64_t Q1,
                                       int32_t c2, int64_t T2, int64_t Q2) {
    const int lane = lane_id();
    const int32_t cnt = a.count[g];
    const bool act = lane < cnt;
    int64_t tv = 0, qv = 0;
    if (act) {
        const int32_t c = r * a.D + a.slots[g * a.D + lane];
        if (c == c1) {
            tv = T1;
            qv = Q1;
        } else if (c == c2) {
            tv = T2;
            qv = Q2;
        } else {
            tv = T[c];
            qv = Q[c];
        }
    }
    int64_t A = 0;
    for (int s = 0; s < a.S; ++s) {
        const int64_t cost = act ? a.alpha[s] * tv + a.beta[s] * qv : LLONG_MIN;
        A += wave_max(cost);
    }
    return A;
}



}  // namespace rp
