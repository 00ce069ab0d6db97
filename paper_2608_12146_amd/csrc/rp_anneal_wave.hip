// Fixed-row population annealing (Alg. 3), one wave per population member.
//
// A member's small state lives in LDS for the whole level: cell of every
// sample and the member pool sorted by (cell, id) as uint16, cell start
// offsets, cell token sums T (int32) and squared sums Q2 (int64), the
// attention weight of every cell (sum_s cost_s), and the inclusive prefix of
// J over row-shards.  J, A and U are held in the wave's registers.  The
// row-shard tables W stay in the member's slab in HBM: only an evaluated
// move touches them (two rows of L*P int32).
//
// Proposal screening is lane-parallel: lane x draws the Philox words of
// proposal k0 + x and resolves its GuidedProposal (binary searches over the
// prefix of J, the cell roulette, member lookups) and its feasibility
// against the current state.  The wave then evaluates, in order, the first
// feasible proposal.  A rejected proposal leaves the state unchanged, so the
// remaining screens stay valid; an accepted one changes it, and the
// remaining proposals of the batch are screened again.  The sequence of
// evaluated proposals, accept decisions and states is therefore exactly the
// sequential one.
//
// Members of a level are updated in place in their slabs (slab_of[m] names
// the slab of member m); resampling hands each parent's slab to its first
// child and copies it for the others (k_copy_slabs).
#include "rp_anneal.h"

// Optional per-phase cycle counters (prologue, screening, evaluation, the
// W-row part of it, commit, epilogue, total, evaluated moves), compiled in
// only with -DRP_PHASE_TIMERS; they take no decision and skip no work.
#ifdef RP_PHASE_TIMERS
#define RP_T_DECL unsigned long long rp_t[8] = {0, 0, 0, 0, 0, 0, 0, 0}, rp_t0 = clock64(), rp_ts = 0;
#define RP_T_BEGIN rp_ts = clock64();
#define RP_T_END(k) rp_t[k] += clock64() - rp_ts;
#define RP_T_FLUSH(m, n)                                                                    \
    if (a.phase_cycles && lane_id() == 0) {                                                 \
        rp_t[6] = clock64() - rp_t0;                                                        \
        rp_t[7] = (unsigned long long)(n);                                                  \
        for (int q_ = 0; q_ < 8; ++q_) atomicAdd(a.phase_cycles + (int64_t)(m) * 8 + q_, rp_t[q_]); \
    }
#else
#define RP_T_DECL
#define RP_T_BEGIN
#define RP_T_END(k)
#define RP_T_FLUSH(m, n)
#endif

namespace rp {

__device__ inline void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

struct MemberLds {
    uint16_t *cell, *pool, *start;
    int32_t *T;
    int64_t *Q;
    int64_t *cpre;  // per cell: inclusive prefix of sum_s cost_s over its row-shard's cells, slot order
    int64_t *Jpre;  // inclusive prefix of J over row-shards
};

// first h in [0, n) with pre[h] > pick (pre non-decreasing, pick < pre[n-1])
__device__ inline int32_t first_above(const int64_t *pre, int32_t n, uint64_t pick) {
    int32_t lo = 0, hi = n - 1;
    while (lo < hi) {
        const int32_t mid = (lo + hi) >> 1;
        if ((uint64_t)pre[mid] > pick) hi = mid;
        else lo = mid + 1;
    }
    return lo;
}
// first h with (h+1)(s2+1) - pre[h] > pick: the prefix of the target
// weights s2 - J_h + 1
__device__ inline int32_t first_target(const int64_t *pre, int32_t n, int64_t s2, uint64_t pick) {
    int32_t lo = 0, hi = n - 1;
    while (lo < hi) {
        const int32_t mid = (lo + hi) >> 1;
        const int64_t v = (int64_t)(mid + 1) * (s2 + 1) - pre[mid];
        if ((uint64_t)v > pick) hi = mid;
        else lo = mid + 1;
    }
    return lo;
}

struct Screen {
    int32_t i, j, c1, c2, pos_i, pos_j, ti, tj;
    bool feas;
};

// Resolves one proposal from its words against the member's current state.
__device__ inline Screen screen_one(const AnnealArgs &a, const MemberLds &M, const int32_t *tv,
                                    const int32_t *s_slots, const int32_t *s_count, uint64_t w0,
                                    uint64_t w1, uint64_t w2, uint64_t w3, uint64_t w4, uint64_t w5,
                                    uint64_t w6, int64_t s1, int64_t s2) {
    Screen sc;
    const int32_t N = a.N, B = a.B, RG = a.RG, D = a.D, G = a.G;
    const bool guided = (uint32_t)w0 < a.p_guide;
    const bool reloc = (uint32_t)(w0 >> 32) < a.rho;
    sc.j = -1;
    sc.pos_i = -1;
    sc.pos_j = -1;
    if (guided) {
        // The source and target row-shard searches are independent: run
        // them in one loop so their LDS reads overlap.
        const uint64_t pk1 = bounded(w1, (uint64_t)s1);
        const uint64_t pk4 = bounded(w4, (uint64_t)((int64_t)RG * (s2 + 1) - s1));
        int32_t lo1 = 0, hi1 = RG - 1, lo2 = 0, hi2 = RG - 1;
        if (s1 == 0) lo1 = hi1 = (int32_t)bounded(w1, (uint64_t)RG);
        while (lo1 < hi1 || lo2 < hi2) {
            const int32_t m1 = (lo1 + hi1) >> 1, m2 = (lo2 + hi2) >> 1;
            const int64_t p1 = M.Jpre[m1], p2 = M.Jpre[m2];
            if (lo1 < hi1) {
                if ((uint64_t)p1 > pk1) hi1 = m1;
                else lo1 = m1 + 1;
            }
            if (lo2 < hi2) {
                if ((uint64_t)((int64_t)(m2 + 1) * (s2 + 1) - p2) > pk4) hi2 = m2;
                else lo2 = m2 + 1;
            }
        }
        const int32_t h1 = lo1, h2 = lo2;
        const int32_t r1 = h1 / G, g1 = h1 % G, cnt1 = s_count[g1];
        const int32_t r2 = h2 / G, g2 = h2 % G;
        sc.c2 = r2 * D + s_slots[g2 * D + (int32_t)bounded(w5, (uint64_t)s_count[g2])];
        const int32_t *sl1 = s_slots + g1 * D;
        const int64_t *cp = M.cpre + r1 * D;
        const int64_t tot = cp[sl1[cnt1 - 1]];
        int32_t xi;
        if (tot == 0) {
            xi = (int32_t)bounded(w2, (uint64_t)cnt1);
        } else {
            const uint64_t pk = bounded(w2, (uint64_t)tot);
            int32_t lo = 0, hi = cnt1 - 1;
            while (lo < hi) {
                const int32_t mid = (lo + hi) >> 1;
                if ((uint64_t)cp[sl1[mid]] > pk) hi = mid;
                else lo = mid + 1;
            }
            xi = lo;
        }
        sc.c1 = r1 * D + sl1[xi];
        const int32_t st1 = M.start[sc.c1], en1 = M.start[sc.c1 + 1];
        const int32_t st2 = M.start[sc.c2], en2 = M.start[sc.c2 + 1];
        sc.pos_i = clampi(st1 + (int32_t)bounded(w3, (uint64_t)(en1 - st1)), 0, N - 1);
        sc.i = M.pool[sc.pos_i];
        if (!reloc) {
            sc.pos_j = clampi(st2 + (int32_t)bounded(w6, (uint64_t)(en2 - st2)), 0, N - 1);
            sc.j = M.pool[sc.pos_j];
        }
    } else {
        sc.i = (int32_t)bounded(w1, (uint64_t)N);
        sc.c1 = M.cell[sc.i];
        if (!reloc) {
            sc.j = (int32_t)bounded(w4, (uint64_t)N);
            sc.c2 = M.cell[sc.j];
        } else {
            sc.c2 = (int32_t)bounded(w4, (uint64_t)B);
        }
    }
    sc.c1 = clampi(sc.c1, 0, B - 1);
    sc.c2 = clampi(sc.c2, 0, B - 1);
    sc.ti = tv[sc.i];
    sc.tj = sc.j >= 0 ? tv[sc.j] : 0;
    const int64_t T1 = M.T[sc.c1], T2 = M.T[sc.c2];
    const int32_t sz1 = M.start[sc.c1 + 1] - M.start[sc.c1];
    bool f = sc.c1 != sc.c2;
    if (f) {
        if (!reloc) f = (T1 - sc.ti + sc.tj <= a.C) && (T2 - sc.tj + sc.ti <= a.C);
        else f = (sz1 >= 2) && (T2 + sc.ti <= a.C);
    }
    sc.feas = f;
    return sc;
}

__device__ inline int32_t count_less16(const uint16_t *pool, int32_t lo, int32_t hi, int32_t v,
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

// Remove pool[from], insert v at `to`, shifting the elements in between by
// one position (one wave; each chunk's reads complete before its writes).
__device__ inline void pool_move16(uint16_t *pool, int32_t from, int32_t to, int32_t v) {
    const int lane = lane_id();
    if (from < to) {
        for (int32_t base = from; base < to; base += kWave) {
            const int32_t x = base + lane;
            uint16_t val = 0;
            if (x < to) val = pool[x + 1];
            wave_sync();
            if (x < to) pool[x] = val;
            wave_sync();
        }
    } else if (from > to) {
        for (int32_t top = from; top > to; top -= kWave) {
            const int32_t x = top - lane;
            uint16_t val = 0;
            if (x > to) val = pool[x - 1];
            wave_sync();
            if (x > to) pool[x] = val;
            wave_sync();
        }
    }
    if (lane == 0) pool[to] = (uint16_t)v;
    wave_sync();
}

// Attention part of row-shard (r, g) from the LDS cell statistics with up to
// two cells replaced (lanes over the shard's cells).
__device__ inline int64_t attention_lds(const AnnealArgs &a, const MemberLds &M, const int32_t *s_slots,
                                        const int32_t *s_count, int32_t r, int32_t g, int32_t c1,
                                        int64_t T1, int64_t Q1, int32_t c2, int64_t T2, int64_t Q2) {
    const int lane = lane_id();
    const int32_t cnt = s_count[g];
    const bool act = lane < cnt;
    int64_t tv = 0, qv = 0;
    if (act) {
        const int32_t c = r * a.D + s_slots[g * a.D + lane];
        if (c == c1) {
            tv = T1;
            qv = Q1;
        } else if (c == c2) {
            tv = T2;
            qv = Q2;
        } else {
            tv = M.T[c];
            qv = M.Q[c];
        }
    }
    int64_t A = 0;
    for (int s = 0; s < a.S; ++s) A += wave_max(act ? a.alpha[s] * tv + a.beta[s] * qv : LLONG_MIN);
    return A;
}

// cpre of row-shard (r, g): inclusive prefix of the cells' attention weights
// in slot order (lanes over the shard's cells).
__device__ inline void rebuild_cpre(const AnnealArgs &a, const MemberLds &M, const int32_t *s_slots,
                                    const int32_t *s_count, int32_t r, int32_t g) {
    const int lane = lane_id();
    const int32_t cnt = s_count[g];
    int64_t w = 0;
    int32_t c = 0;
    if (lane < cnt) {
        c = r * a.D + s_slots[g * a.D + lane];
        const int64_t t = M.T[c], q = M.Q[c];
        for (int s = 0; s < a.S; ++s) w += a.alpha[s] * t + a.beta[s] * q;
    }
    const int64_t incl = wave_incl_scan(w);
    if (lane < cnt) M.cpre[c] = incl;
}

constexpr int kCh = 8;  // W row chunks (of 64 entries) held in registers per move

// v[h] for a uniform row-shard index h held as lane h % 64 of register h / 64.
template <int JPL>
__device__ inline int64_t lane_get(const int64_t (&v)[JPL], int32_t h) {
    int64_t out = 0;
#pragma unroll
    for (int x = 0; x < JPL; ++x)
        if ((h >> 6) == x) out = (int64_t)readlane64((uint64_t)v[x], h & 63);
    return out;
}

template <int JPL, bool TLDS>
__global__ void __launch_bounds__(512) k_anneal_wave(AnnealArgs a) {
    extern __shared__ char smem[];
    const int lane = lane_id(), wv = wave_id();
    const int32_t N = a.N, B = a.B, RG = a.RG, LP = a.LP, D = a.D, G = a.G, P = a.P;
    int32_t *s_slots = reinterpret_cast<int32_t *>(smem);
    int32_t *s_count = s_slots + G * D;
    int32_t *s_shard = s_count + G;
    int32_t *s_t = s_shard + D;  // [N] when TLDS
    for (int32_t x = threadIdx.x; x < G * D; x += blockDim.x) s_slots[x] = a.slots[x];
    for (int32_t x = threadIdx.x; x < G; x += blockDim.x) s_count[x] = a.count[x];
    for (int32_t x = threadIdx.x; x < D; x += blockDim.x) s_shard[x] = a.slot_shard[x];
    if (TLDS)
        for (int32_t x = threadIdx.x; x < N; x += blockDim.x) s_t[x] = a.t[x];
    __syncthreads();
    const int m = blockIdx.x * a.mpw + wv;
    if (m >= a.pop) return;  // no block barrier follows
    const int32_t *tv = TLDS ? s_t : a.t;
    char *slab = a.slabs + (int64_t)a.slab_of[m] * a.off.bytes;
    char *mine = smem + a.lds_shared + (int64_t)wv * a.lds_member;
    MemberLds M;
    M.cell = reinterpret_cast<uint16_t *>(mine + a.o_cell);
    M.pool = reinterpret_cast<uint16_t *>(mine + a.o_pool);
    M.start = reinterpret_cast<uint16_t *>(mine + a.o_start);
    M.T = reinterpret_cast<int32_t *>(mine + a.o_T);
    M.Q = reinterpret_cast<int64_t *>(mine + a.o_Q);
    M.cpre = reinterpret_cast<int64_t *>(mine + a.o_acost);
    M.Jpre = reinterpret_cast<int64_t *>(mine + a.o_Jpre);
    int32_t *g_cell = at<int32_t>(slab, a.off.cell);
    int32_t *g_pool = at<int32_t>(slab, a.off.pool);
    int32_t *g_start = at<int32_t>(slab, a.off.start);
    int64_t *g_T = at<int64_t>(slab, a.off.T);
    int64_t *g_Q = at<int64_t>(slab, a.off.Q);
    int32_t *W = at<int32_t>(slab, a.off.W);
    int64_t *g_J = at<int64_t>(slab, a.off.J);
    int64_t *g_A = at<int64_t>(slab, a.off.A);

    RP_T_DECL
    RP_T_BEGIN
    // Prologue: member state into LDS and registers.
    {
        // 4 ids per lane and 4 chunks in flight
        const int32_t n4 = N >> 2;
        const int4 *c4 = reinterpret_cast<const int4 *>(g_cell), *p4 = reinterpret_cast<const int4 *>(g_pool);
        ushort4 *lc4 = reinterpret_cast<ushort4 *>(M.cell), *lp4 = reinterpret_cast<ushort4 *>(M.pool);
#pragma unroll 4
        for (int32_t x = lane; x < n4; x += kWave) {
            const int4 u = c4[x], v = p4[x];
            lc4[x] = make_ushort4((uint16_t)u.x, (uint16_t)u.y, (uint16_t)u.z, (uint16_t)u.w);
            lp4[x] = make_ushort4((uint16_t)v.x, (uint16_t)v.y, (uint16_t)v.z, (uint16_t)v.w);
        }
        for (int32_t x = (n4 << 2) + lane; x < N; x += kWave) {
            M.cell[x] = (uint16_t)g_cell[x];
            M.pool[x] = (uint16_t)g_pool[x];
        }
    }
#pragma unroll 4
    for (int32_t x = lane; x <= B; x += kWave) M.start[x] = (uint16_t)g_start[x];
#pragma unroll 4
    for (int32_t x = lane; x < B; x += kWave) {
        M.T[x] = (int32_t)g_T[x];
        M.Q[x] = g_Q[x];
    }
    wave_sync();
    for (int32_t h = lane; h < RG; h += kWave) {  // lanes over row-shards
        const int32_t r = h / G, g = h % G;
        int64_t acc = 0;
        for (int32_t x = 0; x < s_count[g]; ++x) {
            const int32_t c = r * D + s_slots[g * D + x];
            const int64_t t = M.T[c], q = M.Q[c];
            for (int s = 0; s < a.S; ++s) acc += a.alpha[s] * t + a.beta[s] * q;
            M.cpre[c] = acc;
        }
    }
    int64_t Jr[JPL], Ar[JPL];
#pragma unroll
    for (int x = 0; x < JPL; ++x) {
        const int h = x * kWave + lane;
        Jr[x] = h < RG ? g_J[h] : 0;
        Ar[x] = h < RG ? g_A[h] : 0;
    }
    int64_t Ur = 0;
    if (lane < G)
        for (int r = 0; r < a.R; ++r) Ur += g_J[(int64_t)r * G + lane];
    int64_t s0 = wave_max(lane < G ? Ur : LLONG_MIN);
    int64_t s1 = wave_sum(lane < G ? Ur : 0);
    int64_t s2 = LLONG_MIN;
#pragma unroll
    for (int x = 0; x < JPL; ++x)
        if (x * kWave + lane < RG) s2 = Jr[x] > s2 ? Jr[x] : s2;
    s2 = wave_max(s2);
    {
        int64_t carry = 0;
#pragma unroll
        for (int x = 0; x < JPL; ++x) {
            const int h = x * kWave + lane;
            const int64_t incl = wave_incl_scan(h < RG ? Jr[x] : 0) + carry;
            if (h < RG) M.Jpre[h] = incl;
            carry = (int64_t)readlane64((uint64_t)incl, kWave - 1);
        }
    }
    wave_sync();
    int64_t b0 = s0, b1 = s1, b2 = s2;
    int32_t best_is_start = 1;
    int32_t *bl = a.best + (int64_t)m * N;
    // Only a trajectory best strictly below the incumbent at the level start
    // can become the next incumbent, so only such a layout is kept.
    const int64_t x0 = a.xscore[0], x1 = a.xscore[1], x2 = a.xscore[2];
    if (lex_less(s0, s1, s2, x0, x1, x2)) {
        // A start state better than the incumbent is itself a trajectory
        // best; keep its layout, since the slab is updated in place.
        for (int32_t x = lane; x < N; x += kWave) bl[x] = M.cell[x];
        best_is_start = 0;
    }
    RP_T_END(0)
    int64_t n_acc = 0, n_eval = 0;
    double e_cur = energy(s0, s1, s2, a.scale);
    uint8_t *log = a.step_log ? a.step_log + (int64_t)m * a.K : nullptr;
    const int32_t nch = (LP + kWave - 1) / kWave;
    int32_t nva[kCh], nvb[kCh];  // new W values of the evaluated move (first kCh chunks)

    for (int32_t k0 = 0; k0 < a.K; k0 += kWave) {
        const int32_t k = k0 + lane;
        const U64x4 b0w = philox4x64_10((uint64_t)k, (uint64_t)(uint32_t)a.level, (uint64_t)(uint32_t)m, 0,
                                        a.seed, 0);
        const U64x4 b1w = philox4x64_10((uint64_t)k, (uint64_t)(uint32_t)a.level, (uint64_t)(uint32_t)m, 1,
                                        a.seed, 0);
        const uint64_t w0 = b0w.v[0], w1 = b0w.v[1], w2 = b0w.v[2], w3 = b0w.v[3];
        const uint64_t w4 = b1w.v[0], w5 = b1w.v[1], w6 = b1w.v[2], w7 = b1w.v[3];
        uint64_t pending = __ballot(k < a.K);
        RP_T_BEGIN
        Screen sc = screen_one(a, M, tv, s_slots, s_count, w0, w1, w2, w3, w4, w5, w6, s1, s2);
        uint64_t feas = __ballot(sc.feas && k < a.K);
        RP_T_END(1)
        while (pending) {
            const uint64_t cand = pending & feas;
            const uint64_t below = cand ? (cand & (~cand + 1)) - 1 : ~0ull;  // bits below the first candidate
            if (log && ((pending & below) >> lane) & 1ull) log[k] = 0;
            if (!cand) break;
            const int f = first_lane(cand);
            pending &= ~((cand & (~cand + 1)) | below);
            // ---- evaluate proposal f (uniform over the wave)
            RP_T_BEGIN
            const int32_t i = __builtin_amdgcn_readlane(sc.i, f);
            const int32_t j = __builtin_amdgcn_readlane(sc.j, f);
            const int32_t c1 = __builtin_amdgcn_readlane(sc.c1, f);
            const int32_t c2 = __builtin_amdgcn_readlane(sc.c2, f);
            int32_t pos_i = __builtin_amdgcn_readlane(sc.pos_i, f);
            int32_t pos_j = __builtin_amdgcn_readlane(sc.pos_j, f);
            const int64_t ti = __builtin_amdgcn_readlane(sc.ti, f);
            const int64_t tj = __builtin_amdgcn_readlane(sc.tj, f);
            const uint64_t fw0 = readlane64(w0, f), fw7 = readlane64(w7, f);
            const bool reloc = (uint32_t)(fw0 >> 32) < a.rho;
            n_eval += 1;
            const int64_t T1 = M.T[c1], T2 = M.T[c2], Q1 = M.Q[c1], Q2v = M.Q[c2];
            const int64_t nT1 = T1 - ti + tj, nT2 = T2 + ti - tj;
            const int64_t nQ1 = Q1 - ti * ti + tj * tj, nQ2 = Q2v + ti * ti - tj * tj;
            const int32_t ra = c1 / D, ga = s_shard[c1 % D];
            const int32_t rb = c2 / D, gb = s_shard[c2 % D];
            const int32_t ha = ra * G + ga, hb = rb * G + gb;
            const int32_t *qi = a.q + (int64_t)i * LP;
            const int32_t *qj = j >= 0 ? a.q + (int64_t)j * LP : nullptr;
            // Issue the first group of W and q row loads now, so their
            // latency overlaps the attention and score bookkeeping below.
            int32_t xa[kCh], xb[kCh], xi_[kCh], xj[kCh];
            if (ha != hb) {
                const int32_t *Wa = W + (int64_t)ha * LP, *Wb = W + (int64_t)hb * LP;
#pragma unroll
                for (int c = 0; c < kCh; ++c) {
                    const int32_t e = c * kWave + lane;
                    xa[c] = 0; xb[c] = 0; xi_[c] = 0; xj[c] = 0;
                    if (c < nch && e < LP) {
                        xa[c] = Wa[e];
                        xb[c] = Wb[e];
                        xi_[c] = qi[e];
                        xj[c] = qj ? qj[e] : 0;
                    }
                }
            }
            const int64_t Jha = lane_get<JPL>(Jr, ha), Jhb = lane_get<JPL>(Jr, hb), Aha = lane_get<JPL>(Ar, ha);
            int64_t Aa, Ab, Ja, Jb;
            if (ha == hb) {
                Aa = attention_lds(a, M, s_slots, s_count, ra, ga, c1, nT1, nQ1, c2, nT2, nQ2);
                Ab = Aa;
                Ja = Aa + (Jha - Aha);
                Jb = Ja;
            } else {
                Aa = attention_lds(a, M, s_slots, s_count, ra, ga, c1, nT1, nQ1, -1, 0, 0);
                Ab = attention_lds(a, M, s_slots, s_count, rb, gb, c2, nT2, nQ2, -1, 0, 0);
                const int32_t *Wa = W + (int64_t)ha * LP, *Wb = W + (int64_t)hb * LP;
                RP_T_END(2)
                RP_T_BEGIN
                int64_t suma = 0, sumb = 0;
                for (int32_t g0 = 0; g0 < nch; g0 += kCh) {
                    if (g0 > 0) {
#pragma unroll
                        for (int c = 0; c < kCh; ++c) {  // every load of the group in flight at once
                            const int32_t e = (g0 + c) * kWave + lane;
                            xa[c] = 0; xb[c] = 0; xi_[c] = 0; xj[c] = 0;
                            if (g0 + c < nch && e < LP) {
                                xa[c] = Wa[e];
                                xb[c] = Wb[e];
                                xi_[c] = qi[e];
                                xj[c] = qj ? qj[e] : 0;
                            }
                        }
                    }
#pragma unroll
                    for (int c = 0; c < kCh; ++c) {
                        if (g0 + c < nch) {
                            const int32_t e = (g0 + c) * kWave + lane;
                            const int32_t d = xi_[c] - xj[c];
                            const int32_t va = e < LP ? xa[c] - d : INT32_MIN;
                            const int32_t vb = e < LP ? xb[c] + d : INT32_MIN;
                            if (g0 == 0) {
                                nva[c] = va;
                                nvb[c] = vb;
                            }
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
                Ja = Aa + (suma << a.F);
                Jb = Ab + (sumb << a.F);
                RP_T_END(3)
                RP_T_BEGIN
            }
            int64_t Un = Ur;
            if (lane == ga) Un += Ja - Jha;
            if (lane == gb && hb != ha) Un += Jb - Jhb;
            const int64_t n0 = wave_max(lane < G ? Un : LLONG_MIN);
            const int64_t n1 = s1 + (Ja - Jha) + (hb != ha ? (Jb - Jhb) : 0);
            int64_t n2 = LLONG_MIN;
#pragma unroll
            for (int x = 0; x < JPL; ++x) {
                const int h = x * kWave + lane;
                if (h < RG) {
                    const int64_t v = h == ha ? Ja : (h == hb ? Jb : Jr[x]);
                    n2 = v > n2 ? v : n2;
                }
            }
            n2 = wave_max(n2);
            const double e_new = energy(n0, n1, n2, a.scale);
            const double den = fabs(e_cur) > 1.0 ? fabs(e_cur) : 1.0;
            const double delta = (e_new - e_cur) / den;
            const double z = (delta > 0.0 ? delta : 0.0) / a.temp;
            const double u = (double)(uint32_t)(fw7 >> 32) * (1.0 / 4294967296.0);
            const bool accept = lex_less(n0, n1, n2, s0, s1, s2) || (u < exp_det(-z));
            RP_T_END(2)
            if (!accept) {
                if (log && lane == f) log[k] = 1;
                continue;  // the remaining screens stay valid
            }
            if (log && lane == f) log[k] = 2;
            n_acc += 1;
            RP_T_BEGIN
            // ---- commit
            const int32_t st1 = M.start[c1], en1 = M.start[c1 + 1];
            const int32_t st2 = M.start[c2], en2 = M.start[c2 + 1];
            if (pos_i < 0) pos_i = st1 + count_less16(M.pool, st1, en1, i, -1, N);
            int32_t to1, to2 = 0;
            if (!reloc) {
                if (pos_j < 0) pos_j = st2 + count_less16(M.pool, st2, en2, j, -1, N);
                to1 = st1 + count_less16(M.pool, st1, en1, j, i, N);
                to2 = st2 + count_less16(M.pool, st2, en2, i, j, N);
            } else {
                const int32_t rk = count_less16(M.pool, st2, en2, i, -1, N);
                to1 = (c1 < c2) ? (st2 - 1 + rk) : (st2 + rk);
            }
            pos_i = clampi(pos_i, 0, N - 1);
            pos_j = clampi(pos_j, 0, N - 1);
            to1 = clampi(to1, 0, N - 1);
            to2 = clampi(to2, 0, N - 1);
            wave_sync();
            if (ha != hb) {
                int32_t *Wa = W + (int64_t)ha * LP, *Wb = W + (int64_t)hb * LP;
#pragma unroll
                for (int c = 0; c < kCh; ++c) {
                    const int32_t e = c * kWave + lane;
                    if (c < nch && e < LP) {
                        Wa[e] = nva[c];
                        Wb[e] = nvb[c];
                    }
                }
                for (int32_t e = kCh * kWave + lane; e < LP; e += kWave) {
                    const int32_t d = qi[e] - (qj ? qj[e] : 0);
                    Wa[e] -= d;
                    Wb[e] += d;
                }
            }
            if (lane == 0) {
                M.cell[i] = (uint16_t)c2;
                if (j >= 0) M.cell[j] = (uint16_t)c1;
                M.T[c1] = (int32_t)nT1;
                M.Q[c1] = nQ1;
                M.T[c2] = (int32_t)nT2;
                M.Q[c2] = nQ2;
            }
            wave_sync();
            rebuild_cpre(a, M, s_slots, s_count, ra, ga);
            if (hb != ha) rebuild_cpre(a, M, s_slots, s_count, rb, gb);
            if (!reloc) {
                pool_move16(M.pool, pos_i, to1, j);
                pool_move16(M.pool, pos_j, to2, i);
            } else {
                pool_move16(M.pool, pos_i, to1, i);
                if (c1 < c2) {
                    for (int32_t c = c1 + 1 + lane; c <= c2; c += kWave) M.start[c] -= 1;
                } else {
                    for (int32_t c = c2 + 1 + lane; c <= c1; c += kWave) M.start[c] += 1;
                }
            }
            int64_t carry = 0;
#pragma unroll
            for (int x = 0; x < JPL; ++x) {
                const int h = x * kWave + lane;
                if (h == ha) {
                    Jr[x] = Ja;
                    Ar[x] = Aa;
                } else if (h == hb) {
                    Jr[x] = Jb;
                    Ar[x] = Ab;
                }
                const int64_t incl = wave_incl_scan(h < RG ? Jr[x] : 0) + carry;
                if (h < RG) M.Jpre[h] = incl;
                carry = (int64_t)readlane64((uint64_t)incl, kWave - 1);
            }
            Ur = Un;
            s0 = n0;
            s1 = n1;
            s2 = n2;
            e_cur = e_new;
            wave_sync();
            if (lex_less(s0, s1, s2, b0, b1, b2)) {
                b0 = s0;
                b1 = s1;
                b2 = s2;
                best_is_start = 0;
                if (lex_less(s0, s1, s2, x0, x1, x2))
                    for (int32_t x = lane; x < N; x += kWave) bl[x] = M.cell[x];
            }
            RP_T_END(4)
            if (pending) {
                RP_T_BEGIN
                sc = screen_one(a, M, tv, s_slots, s_count, w0, w1, w2, w3, w4, w5, w6, s1, s2);
                feas = __ballot(sc.feas && k < a.K);
                RP_T_END(1)
            }
        }
    }
    // Epilogue: the terminal state back to the slab.
    RP_T_BEGIN
    wave_sync();
    for (int32_t x = lane; x < N; x += kWave) {
        g_cell[x] = M.cell[x];
        g_pool[x] = M.pool[x];
    }
    for (int32_t x = lane; x <= B; x += kWave) g_start[x] = M.start[x];
    for (int32_t x = lane; x < B; x += kWave) {
        g_T[x] = M.T[x];
        g_Q[x] = M.Q[x];
    }
#pragma unroll
    for (int x = 0; x < JPL; ++x) {
        const int h = x * kWave + lane;
        if (h < RG) {
            g_J[h] = Jr[x];
            g_A[h] = Ar[x];
        }
    }
    if (lane == 0) {
        int64_t *res = a.results + (int64_t)m * kRes;
        res[0] = s0; res[1] = s1; res[2] = s2;
        res[3] = b0; res[4] = b1; res[5] = b2;
        res[6] = n_acc; res[7] = n_eval;
        res[8] = best_is_start;
        res[9] = m;
    }
    RP_T_END(5)
    RP_T_FLUSH(m, n_eval)
}

// Copies the slab of each duplicated parent into the slab its extra child
// takes over (entries 0 .. n_copies-1 of src/dst).  Each copy is split over
// kCopySplit workgroups, four 16-byte loads in flight per thread.
constexpr int kCopySplit = 8;
__global__ void __launch_bounds__(256) k_copy_slabs(char *slabs, int64_t bytes, const int32_t *src,
                                                    const int32_t *dst, const int32_t *n_copies) {
    const int b = blockIdx.x / kCopySplit, part = blockIdx.x % kCopySplit;
    if (b >= *n_copies) return;
    const int64_t n16 = bytes / 16;
    const int64_t per = (n16 + kCopySplit - 1) / kCopySplit;
    const int64_t lo = part * per, hi = lo + per < n16 ? lo + per : n16;
    const int4 *s = reinterpret_cast<const int4 *>(slabs + (int64_t)src[b] * bytes);
    int4 *d = reinterpret_cast<int4 *>(slabs + (int64_t)dst[b] * bytes);
    const int64_t step = blockDim.x;
    int64_t x = lo + threadIdx.x;
    for (; x + 3 * step < hi; x += 4 * step) {
        const int4 v0 = s[x], v1 = s[x + step], v2 = s[x + 2 * step], v3 = s[x + 3 * step];
        d[x] = v0;
        d[x + step] = v1;
        d[x + 2 * step] = v2;
        d[x + 3 * step] = v3;
    }
    for (; x < hi; x += step) d[x] = s[x];
}

// Chooses the wave kernel's launch shape; returns false when a member's
// state does not fit LDS (the caller then uses the workgroup kernel).
bool wave_plan(AnnealArgs &a, int32_t n_cu, int32_t *mpw_out, bool *tlds_out) {
    if (a.N > 65535 || a.B + 1 > 65535 || a.C > 2147483647LL || a.RG > kWave * 8) return false;
    auto up8 = [](int64_t x) { return (x + 7) & ~(int64_t)7; };
    int64_t o = 0;
    a.o_cell = (int32_t)o; o = up8(o + 2 * (int64_t)a.N);
    a.o_pool = (int32_t)o; o = up8(o + 2 * (int64_t)a.N);
    a.o_start = (int32_t)o; o = up8(o + 2 * ((int64_t)a.B + 1));
    a.o_T = (int32_t)o; o = up8(o + 4 * (int64_t)a.B);
    a.o_Q = (int32_t)o; o = up8(o + 8 * (int64_t)a.B);
    a.o_acost = (int32_t)o; o = up8(o + 8 * (int64_t)a.B);
    a.o_Jpre = (int32_t)o; o = up8(o + 8 * (int64_t)a.RG);
    const int64_t member = o;
    const int64_t lim = 160 * 1024;
    const int64_t base = up8(4 * ((int64_t)a.G * a.D + a.G + a.D));
    const int64_t with_t = up8(base + 4 * (int64_t)a.N);
    const int64_t cap_g = (lim - base) / member, cap_t = (lim - with_t) / member;
    if (cap_g < 1) return false;
    // One member per wave, spread over every CU before any CU takes more:
    // ceil(pop / CUs) members per workgroup, within LDS and 8 waves.
    int64_t want = ((int64_t)a.pop + n_cu - 1) / n_cu;
    want = want < 1 ? 1 : (want > 8 ? 8 : want);
    bool tlds = cap_t >= want;
    int64_t mpw = tlds ? want : (cap_g < want ? cap_g : want);
    a.mpw = (int32_t)mpw;
    a.lds_shared = (int32_t)(tlds ? with_t : base);
    a.lds_member = (int32_t)member;
    *mpw_out = a.mpw;
    *tlds_out = tlds;
    return true;
}

template <int JPL, bool TLDS>
static int launch_t(const AnnealArgs &a, hipStream_t stream) {
    const size_t lds = (size_t)a.lds_shared + (size_t)a.mpw * a.lds_member;
    static_assert(JPL >= 1, "");
    if (hipFuncSetAttribute((const void *)k_anneal_wave<JPL, TLDS>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
        return ROUTEPACK_E_DEVICE;
    const unsigned grid = (unsigned)((a.pop + a.mpw - 1) / a.mpw);
    hipLaunchKernelGGL((k_anneal_wave<JPL, TLDS>), dim3(grid), dim3(kWave * a.mpw), lds, stream, a);
    return hipGetLastError() == hipSuccess ? ROUTEPACK_OK : ROUTEPACK_E_DEVICE;
}

int launch_anneal_wave(const AnnealArgs &a, bool tlds, hipStream_t stream) {
    const int jpl = (a.RG + kWave - 1) / kWave;
    if (jpl <= 1) return tlds ? launch_t<1, true>(a, stream) : launch_t<1, false>(a, stream);
    if (jpl <= 2) return tlds ? launch_t<2, true>(a, stream) : launch_t<2, false>(a, stream);
    return tlds ? launch_t<8, true>(a, stream) : launch_t<8, false>(a, stream);
}

int launch_copy_slabs(char *slabs, int64_t bytes, const int32_t *src, const int32_t *dst,
                      const int32_t *n_copies, int32_t pop, hipStream_t stream) {
    hipLaunchKernelGGL(k_copy_slabs, dim3(pop * kCopySplit), dim3(256), 0, stream, slabs, bytes, src, dst,
                       n_copies);
    return hipGetLastError() == hipSuccess ? ROUTEPACK_OK : ROUTEPACK_E_DEVICE;
}

}  // namespace rp
