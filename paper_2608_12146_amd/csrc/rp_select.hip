// QualityDiversitySelect (arXiv 2608.12146, Sec. 4.1.1 "Diverse Fixed-Row
// Seeding"; Alg. 2, the selection before the cyclic fill; cost in Sec. 4.2):
// orders canonical-distinct candidate layouts greedily from the exact-score
// winner by the smallest distance to those already chosen minus the
// normalised primary-score gap.  The distance adds cell and row
// co-assignment to a Sliced-Wasserstein sketch of the row features (the
// sorted projections of the row-feature matrix on fixed directions).
//
// Every quantity is an integer: row features in fixed point, sign-vector
// directions, and the comparison of (distance - gap) cross-multiplied in
// 128 bits, so the order is exact.  Kernels:
//   k_cell_stats   per candidate: sample count and smallest member of each
//                  cell and each row (the co-assignment tests need them)
//   k_row_sketch   per (row, candidate): the row's token moments and
//                  per-layer EDP-load profile, its fixed-point features and
//                  their projections on the QDS_Q directions
//   k_sort_proj    per (direction, candidate): the projections sorted
//   k_pair_dist    per candidate pair: the distance numerator
//   k_greedy       one wave: the selection order
//   k_fill         the population, the order repeated
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "routepack.h"
#include "rp_device.h"
#include "rp_internal.h"

namespace rp {
namespace {

constexpr int kQ = 8;            // projection directions
constexpr int kFrac = 20;        // fractional bits of the row features
constexpr uint64_t kTag = 4;     // Philox counter tag of the directions
constexpr int kThreads = 256;
constexpr int kMaxCand = 64;
constexpr int kChunk = 2048;     // members of a row gathered per pass

struct SelArgs {
    int32_t N, L, P, D, G, R, M, F, B;
    int64_t C, k;
    uint64_t seed;
    const int32_t *t, *q, *cand, *shard;   // shard: [D] EDP shard of each slot
    int32_t *csize, *cmin, *rsize, *rmin;  // [M][B], [M][B], [M][R], [M][R]
    unsigned long long *ctok;              // [M][B] tokens of each cell
    int64_t *proj;                         // [M][kQ][R]
    int64_t *dist;                         // [M][M] distance numerators
    int32_t *bad;                          // set when a candidate holds an id outside [0, B)
};

__global__ void __launch_bounds__(kThreads) k_cell_stats(SelArgs s) {
    const int m = blockIdx.x;
    const int32_t *x = s.cand + (int64_t)m * s.N;
    int32_t *cs = s.csize + (int64_t)m * s.B, *cm = s.cmin + (int64_t)m * s.B;
    int32_t *rs = s.rsize + (int64_t)m * s.R, *rm = s.rmin + (int64_t)m * s.R;
    unsigned long long *ct = s.ctok + (int64_t)m * s.B;
    for (int32_t c = threadIdx.x; c < s.B; c += blockDim.x) {
        cs[c] = 0;
        cm[c] = INT32_MAX;
        ct[c] = 0;
    }
    for (int32_t r = threadIdx.x; r < s.R; r += blockDim.x) {
        rs[r] = 0;
        rm[r] = INT32_MAX;
    }
    __syncthreads();
    for (int32_t i = threadIdx.x; i < s.N; i += blockDim.x) {
        const int32_t c = x[i];
        if (c < 0 || c >= s.B) {
            atomicOr(s.bad, 1);
            continue;
        }
        atomicAdd(cs + c, 1);
        atomicMin(cm + c, i);
        atomicAdd(ct + c, (unsigned long long)s.t[i]);
        atomicAdd(rs + c / s.D, 1);
        atomicMin(rm + c / s.D, i);
    }
    __syncthreads();
    // a candidate must be a layout: every cell non-empty and within capacity
    for (int32_t c = threadIdx.x; c < s.B; c += blockDim.x)
        if (cs[c] == 0 || ct[c] > (unsigned long long)s.C) atomicOr(s.bad, 1);
}

// One workgroup per (row r, candidate m): T, sum t^2 and, per layer, the sum
// over shards of the largest rank load W(r, g, l, p); then the fixed-point
// features h and their projections on the directions.
__global__ void __launch_bounds__(kThreads) k_row_sketch(SelArgs s) {
    const int32_t r = blockIdx.x, m = blockIdx.y;
    const int tid = threadIdx.x;
    const int32_t *x = s.cand + (int64_t)m * s.N;
    const int32_t LP = s.L * s.P, GLP = s.G * LP;
    extern __shared__ __align__(16) char smem[];
    int64_t *acc = reinterpret_cast<int64_t *>(smem);          // [G][L][P]
    int64_t *hf = acc + GLP;                                    // [F]
    int32_t *mem = reinterpret_cast<int32_t *>(hf + s.F);       // [kChunk] member | shard << 16
    __shared__ int32_t s_n;
    __shared__ unsigned long long s_T, s_Q;
    for (int32_t e = tid; e < GLP; e += kThreads) acc[e] = 0;
    if (tid == 0) {
        s_T = 0;
        s_Q = 0;
    }
    uint64_t T = 0, Q = 0;
    for (int32_t base = 0; base < s.N; base += kChunk) {
        if (tid == 0) s_n = 0;
        __syncthreads();
        const int32_t top = base + kChunk < s.N ? base + kChunk : s.N;
        for (int32_t i = base + tid; i < top; i += kThreads) {
            const int32_t c = x[i];
            if (c / s.D == r) {
                const int32_t slot = atomicAdd(&s_n, 1);
                mem[slot] = i | (s.shard[c - r * s.D] << 16);
                const uint64_t ti = (uint64_t)s.t[i];
                T += ti;
                Q += ti * ti;
            }
        }
        __syncthreads();
        const int32_t n = s_n;
        for (int32_t e = tid; e < GLP; e += kThreads) {
            const int32_t g = e / LP, lp = e - g * LP;
            int64_t a = 0;
            for (int32_t u = 0; u < n; ++u) {
                const int32_t v = mem[u];
                if ((v >> 16) == g) a += s.q[(int64_t)(v & 0xFFFF) * LP + lp];
            }
            acc[e] += a;
        }
        __syncthreads();
    }
    atomicAdd(&s_T, (unsigned long long)T);
    atomicAdd(&s_Q, (unsigned long long)Q);
    __syncthreads();
    const int64_t DC = (int64_t)s.D * s.C;
    if (tid == 0) {
        hf[0] = (int64_t)(((unsigned __int128)s_T << kFrac) / (uint64_t)DC);
        hf[1] = (int64_t)(((unsigned __int128)s_Q << kFrac) / ((unsigned __int128)DC * (uint64_t)s.C));
    }
    for (int32_t l = tid; l < s.L; l += kThreads) {
        int64_t E = 0;
        for (int32_t g = 0; g < s.G; ++g) {
            int64_t mx = 0;
            for (int32_t p = 0; p < s.P; ++p) {
                const int64_t v = acc[(int64_t)g * LP + l * s.P + p];
                mx = v > mx ? v : mx;
            }
            E += mx;
        }
        hf[2 + l] = (int64_t)(((unsigned __int128)E << kFrac) / (uint64_t)(s.k * DC));
    }
    __syncthreads();
    if (tid < kQ) {
        const U64x4 blk = philox4x64_10((uint64_t)tid, 0, 0, kTag, s.seed, 0);
        int64_t v = 0;
        for (int32_t f = 0; f < s.F; ++f) {
            const bool plus = (blk.v[f >> 6] >> (f & 63)) & 1;
            v += plus ? hf[f] : -hf[f];
        }
        s.proj[((int64_t)m * kQ + tid) * s.R + r] = v;
    }
}

// One workgroup per (direction k, candidate m): the R projections sorted
// ascending, by rank (ties by row index; equal values are interchangeable).
__global__ void __launch_bounds__(kThreads) k_sort_proj(SelArgs s, int64_t *sorted) {
    const int64_t *v = s.proj + ((int64_t)blockIdx.y * kQ + blockIdx.x) * s.R;
    int64_t *out = sorted + ((int64_t)blockIdx.y * kQ + blockIdx.x) * s.R;
    for (int32_t a = threadIdx.x; a < s.R; a += blockDim.x) {
        const int64_t va = v[a];
        int32_t rank = 0;
        for (int32_t b = 0; b < s.R; ++b) {
            const int64_t vb = v[b];
            rank += (vb < va || (vb == va && b < a)) ? 1 : 0;
        }
        out[rank] = va;
    }
}

__device__ inline int64_t block_sum64(int64_t v, int64_t *red) {
    v = wave_sum(v);
    const int lane = lane_id(), wv = wave_id();
    __syncthreads();
    if (lane == 0) red[wv] = v;
    __syncthreads();
    int64_t t = 0;
    for (int w = 0; w < (int)(blockDim.x / kWave); ++w) t += red[w];
    return t;
}

// One workgroup per candidate pair (a, b), a < b: samples whose cell (row)
// sample set differs -- a group of a is unchanged when all of its members
// sit in one group of b of the same size -- and the L1 distance of the
// sorted projections; distance numerator 3 N q R 2^frac d(a, b).
__global__ void __launch_bounds__(kThreads) k_pair_dist(SelArgs s, const int64_t *sorted) {
    int32_t a = 0, rem = blockIdx.x;
    while (rem >= s.M - 1 - a) {
        rem -= s.M - 1 - a;
        ++a;
    }
    const int32_t b = a + 1 + rem;
    const int32_t *xa = s.cand + (int64_t)a * s.N, *xb = s.cand + (int64_t)b * s.N;
    const int32_t *csa = s.csize + (int64_t)a * s.B, *cma = s.cmin + (int64_t)a * s.B;
    const int32_t *csb = s.csize + (int64_t)b * s.B;
    const int32_t *rsa = s.rsize + (int64_t)a * s.R, *rma = s.rmin + (int64_t)a * s.R;
    const int32_t *rsb = s.rsize + (int64_t)b * s.R;
    extern __shared__ __align__(16) char smem[];
    uint32_t *cbroken = reinterpret_cast<uint32_t *>(smem);                 // [B] bits
    uint32_t *rbroken = cbroken + ((s.B + 31) >> 5);                       // [R] bits
    __shared__ int64_t red[kThreads / kWave];
    const int32_t nwc = (s.B + 31) >> 5, nwr = (s.R + 31) >> 5;
    for (int32_t w = threadIdx.x; w < nwc + nwr; w += blockDim.x) cbroken[w] = 0;
    __syncthreads();
    for (int32_t i = threadIdx.x; i < s.N; i += blockDim.x) {
        const int32_t ca = xa[i], cb = xb[i];
        const int32_t ra = ca / s.D, rb = cb / s.D;
        if (cb != xb[cma[ca]] || csb[cb] != csa[ca]) atomicOr(cbroken + (ca >> 5), 1u << (ca & 31));
        if (rb != xb[rma[ra]] / s.D || rsb[rb] != rsa[ra]) atomicOr(rbroken + (ra >> 5), 1u << (ra & 31));
    }
    __syncthreads();
    int64_t changed = 0;
    for (int32_t i = threadIdx.x; i < s.N; i += blockDim.x) {
        const int32_t ca = xa[i], ra = ca / s.D;
        changed += (cbroken[ca >> 5] >> (ca & 31)) & 1;
        changed += (rbroken[ra >> 5] >> (ra & 31)) & 1;
    }
    int64_t e = 0;
    const int64_t *pa = sorted + (int64_t)a * kQ * s.R, *pb = sorted + (int64_t)b * kQ * s.R;
    for (int32_t u = threadIdx.x; u < kQ * s.R; u += blockDim.x) {
        const int64_t d = pa[u] - pb[u];
        e += d < 0 ? -d : d;
    }
    const int64_t AB = block_sum64(changed, red);
    const int64_t E = block_sum64(e, red);
    if (threadIdx.x == 0) {
        const int64_t num = AB * kQ * (int64_t)s.R * ((int64_t)1 << kFrac) + E * s.N;
        s.dist[(int64_t)a * s.M + b] = num;
        s.dist[(int64_t)b * s.M + a] = num;
    }
}

// One wave: lane m holds candidate m's smallest distance numerator to the
// chosen set; each step takes the largest (d_min - gap) * den * s0(x_0),
// the lowest index on a tie.
__global__ void __launch_bounds__(kWave) k_greedy(SelArgs s, const int64_t *primary, int32_t *order) {
    const int m = lane_id();
    const bool live = m < s.M;
    const __int128 den = (__int128)3 * s.N * kQ * s.R * ((int64_t)1 << kFrac);
    const int64_t sw = primary[0];
    const int64_t sm = live ? primary[m] : 0;
    int64_t dmin = live ? s.dist[m] : 0;  // row 0: distances to the winner
    bool left = live && m > 0;
    if (m == 0) order[0] = 0;
    for (int32_t step = 1; step < s.M; ++step) {
        const __int128 key = sw > 0 ? (__int128)dmin * sw - (__int128)(sm - sw) * den : (__int128)dmin;
        // wave argmax of (key, -m) over the candidates still left
        __int128 bk = key;
        int bm = left ? m : kMaxCand;
        for (int off = 1; off < kWave; off <<= 1) {
            const uint64_t lo = __shfl_xor((unsigned long long)(uint64_t)bk, off, kWave);
            const uint64_t hi = __shfl_xor((unsigned long long)(uint64_t)((unsigned __int128)bk >> 64), off, kWave);
            const int om = __shfl_xor(bm, off, kWave);
            const __int128 ok = (__int128)(((unsigned __int128)hi << 64) | lo);
            const bool take = om < kMaxCand && (bm >= kMaxCand || ok > bk || (ok == bk && om < bm));
            if (take) {
                bk = ok;
                bm = om;
            }
        }
        const int best = __builtin_amdgcn_readfirstlane(bm);
        if (m == 0) order[step] = best;
        if (m == best) left = false;
        if (left) {
            const int64_t d = s.dist[(int64_t)best * s.M + m];
            dmin = d < dmin ? d : dmin;
        }
    }
}

__global__ void k_fill(const int32_t *cand, const int32_t *order, int32_t M, int32_t N, int32_t *population) {
    const int32_t p = blockIdx.x;
    const int32_t *src = cand + (int64_t)order[p % M] * N;
    int32_t *dst = population + (int64_t)p * N;
    for (int32_t i = threadIdx.x; i < N; i += blockDim.x) dst[i] = src[i];
}

}  // namespace
}  // namespace rp

using namespace rp;

extern "C" int routepack_select_population(const routepack_problem *prob, const int32_t *lengths,
                                           const int32_t *q, int32_t n_rows, int32_t n_cand,
                                           const int32_t *candidates, const int64_t *primary, uint64_t seed,
                                           int32_t pop_size, int32_t *order, int32_t *population,
                                           hipStream_t stream) {
    Topology topo;
    RP_TRY(check_problem(prob, &topo));
    if (n_rows < 1 || n_cand < 1 || n_cand > kMaxCand || pop_size < 0) return ROUTEPACK_E_INVALID;
    if (!lengths || (!q && prob->n_layers > 0) || !candidates || !primary || !order ||
        (!population && pop_size > 0))
        return ROUTEPACK_E_INVALID;
    const int64_t B64 = (int64_t)n_rows * prob->n_dp, LP = (int64_t)prob->n_layers * prob->n_ranks;
    const int64_t F = 2 + (int64_t)prob->n_layers;
    if (prob->n_samples > 65535 || B64 > 65535 || n_rows > 4096 || F > 256 || prob->n_edp > 32767)
        return ROUTEPACK_E_UNSUPPORTED;
    const int64_t sketch_lds = 8 * ((int64_t)prob->n_edp * LP + F) + 4 * kChunk;
    const int64_t pair_lds = 4 * (((B64 + 31) >> 5) + ((n_rows + 31) >> 5));
    if (sketch_lds > 160 * 1024 || pair_lds > 160 * 1024) return ROUTEPACK_E_UNSUPPORTED;
    // fixed point: a row's sum of squared lengths (at most D C^2) and the
    // features and distance numerators stay within int64
    const int64_t C = prob->capacity;
    if (C > ((int64_t)1 << 31) || (__int128)prob->n_dp * C * C >= ((__int128)1 << 62)) return ROUTEPACK_E_OVERFLOW;
    Scratch scr(stream);
    DeviceProblem dp;
    RP_TRY(upload_problem(prob, topo, scr, &dp, stream));
    const int32_t M = n_cand, N = prob->n_samples, R = n_rows, B = (int32_t)B64;
    SelArgs s{};
    s.N = N; s.L = prob->n_layers; s.P = prob->n_ranks; s.D = prob->n_dp; s.G = prob->n_edp;
    s.R = R; s.M = M; s.F = (int32_t)F; s.B = B;
    s.C = C; s.k = prob->top_k; s.seed = seed;
    s.t = lengths; s.q = q; s.cand = candidates; s.shard = dp.slot_shard;
    s.csize = scr.get<int32_t>((size_t)M * B);
    s.cmin = scr.get<int32_t>((size_t)M * B);
    s.rsize = scr.get<int32_t>((size_t)M * R);
    s.rmin = scr.get<int32_t>((size_t)M * R);
    s.ctok = scr.get<unsigned long long>((size_t)M * B);
    s.proj = scr.get<int64_t>((size_t)M * kQ * R);
    int64_t *sorted = scr.get<int64_t>((size_t)M * kQ * R);
    s.dist = scr.get<int64_t>((size_t)M * M);
    s.bad = scr.get<int32_t>(1);
    if (scr.failed()) return ROUTEPACK_E_DEVICE;
    if (s.k < 1) return ROUTEPACK_E_INVALID;
    RP_HIP(hipMemsetAsync(s.bad, 0, sizeof(int32_t), stream));
    RP_HIP(hipMemsetAsync(s.dist, 0, sizeof(int64_t) * (size_t)M * M, stream));
    hipLaunchKernelGGL(k_cell_stats, dim3(M), dim3(kThreads), 0, stream, s);
    RP_HIP(hipGetLastError());
    int32_t bad = 0;
    RP_HIP(hipMemcpyAsync(&bad, s.bad, sizeof(bad), hipMemcpyDeviceToHost, stream));
    RP_HIP(hipStreamSynchronize(stream));
    if (bad) return ROUTEPACK_E_LAYOUT;  // an id outside [0, R D), an empty or over-full cell
    hipLaunchKernelGGL(k_row_sketch, dim3(R, M), dim3(kThreads), (size_t)sketch_lds, stream, s);
    RP_HIP(hipGetLastError());
    hipLaunchKernelGGL(k_sort_proj, dim3(kQ, M), dim3(kThreads), 0, stream, s, sorted);
    RP_HIP(hipGetLastError());
    if (M > 1) {
        hipLaunchKernelGGL(k_pair_dist, dim3(M * (M - 1) / 2), dim3(kThreads), (size_t)pair_lds, stream, s,
                           (const int64_t *)sorted);
        RP_HIP(hipGetLastError());
    }
    hipLaunchKernelGGL(k_greedy, dim3(1), dim3(kWave), 0, stream, s, primary, order);
    RP_HIP(hipGetLastError());
    if (pop_size > 0) {
        hipLaunchKernelGGL(k_fill, dim3(pop_size), dim3(kThreads), 0, stream, candidates, order, M, N, population);
        RP_HIP(hipGetLastError());
    }
    RP_HIP(hipStreamSynchronize(stream));
    return ROUTEPACK_OK;
}
