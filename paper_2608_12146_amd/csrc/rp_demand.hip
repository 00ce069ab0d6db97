// Window demand aggregation (Sec. 3.3), layer-local LPT placement (Alg. 1)
// and the physical-rank projection (Eq. physical-rank-demand) on gfx950.
//
// Aggregation is an HBM stream: the [N][L*E] int32 demand matrix is reduced
// over its rows.  Each thread owns 4 consecutive columns (one 16-byte load
// per row, so a wave reads 1 KiB contiguous per row) and a contiguous band of
// rows, accumulating in int64 registers; the band partials meet in int64
// atomics, which are exact and order-independent.
#include "rp_device.h"
#include "rp_internal.h"

namespace rp {

__global__ void k_fill_i64(int64_t *p, int64_t n, int64_t v) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

template <int VEC>
__global__ void __launch_bounds__(256) k_aggregate(const int32_t *__restrict__ demand,
                                                   int64_t *__restrict__ agg, int64_t n_rows,
                                                   int64_t n_cols, int64_t rows_per_band) {
    const int64_t col = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * VEC;
    if (col >= n_cols) return;
    const int64_t r0 = (int64_t)blockIdx.y * rows_per_band;
    int64_t r1 = r0 + rows_per_band;
    if (r1 > n_rows) r1 = n_rows;
    int64_t acc[VEC];
#pragma unroll
    for (int c = 0; c < VEC; ++c) acc[c] = 0;
    if (VEC == 4 && col + 4 <= n_cols) {
        const int32_t *p = demand + r0 * n_cols + col;
        int64_t r = r0;
        for (; r + 4 <= r1; r += 4) {
            const int4 a = *reinterpret_cast<const int4 *>(p);
            const int4 b = *reinterpret_cast<const int4 *>(p + n_cols);
            const int4 c = *reinterpret_cast<const int4 *>(p + 2 * n_cols);
            const int4 d = *reinterpret_cast<const int4 *>(p + 3 * n_cols);
            acc[0] += (int64_t)a.x + b.x + c.x + d.x;
            acc[1 % VEC] += (int64_t)a.y + b.y + c.y + d.y;
            acc[2 % VEC] += (int64_t)a.z + b.z + c.z + d.z;
            acc[3 % VEC] += (int64_t)a.w + b.w + c.w + d.w;
            p += 4 * n_cols;
        }
        for (; r < r1; ++r) {
            const int4 a = *reinterpret_cast<const int4 *>(p);
            acc[0] += a.x;
            acc[1 % VEC] += a.y;
            acc[2 % VEC] += a.z;
            acc[3 % VEC] += a.w;
            p += n_cols;
        }
    } else {
        for (int64_t r = r0; r < r1; ++r)
            for (int c = 0; c < VEC; ++c)
                if (col + c < n_cols) acc[c] += demand[r * n_cols + col + c];
    }
#pragma unroll
    for (int c = 0; c < VEC; ++c)
        if (col + c < n_cols && acc[c] != 0)
            atomicAdd(reinterpret_cast<unsigned long long *>(agg + col + c),
                      (unsigned long long)acc[c]);
}

// Layer-local LPT (Alg. 1), one layer per workgroup of one wave.
// Experts are ranked by (-L_{l,e}, e) (ranking by counting: the rank of e
// is the number of experts that precede it), then E greedy steps each pick
// the rank minimising (G_p, p) among ranks with fewer than H experts.
__global__ void __launch_bounds__(64) k_lpt_place(const int64_t *__restrict__ agg, int32_t E,
                                                  int32_t P, int32_t *__restrict__ slot_of,
                                                  int64_t *__restrict__ rank_load,
                                                  int32_t *__restrict__ expert_at_slot) {
    extern __shared__ char smem[];
    int64_t *Ll = reinterpret_cast<int64_t *>(smem);           // [E]
    int64_t *G = Ll + E;                                          // [P]
    int32_t *order = reinterpret_cast<int32_t *>(G + P);          // [E]
    int32_t *nfill = order + E;                                   // [P]
    const int l = blockIdx.x, lane = lane_id();
    const int32_t H = E / P;
    for (int e = lane; e < E; e += kWave) Ll[e] = agg[(int64_t)l * E + e];
    for (int p = lane; p < P; p += kWave) {
        G[p] = 0;
        nfill[p] = 0;
    }
    __syncthreads();
    for (int e = lane; e < E; e += kWave) {
        const int64_t v = Ll[e];
        int32_t rank = 0;
        for (int f = 0; f < E; ++f) {
            const int64_t w = Ll[f];
            rank += (w > v) || (w == v && f < e);
        }
        order[rank] = e;
    }
    __syncthreads();
    for (int k = 0; k < E; ++k) {
        const int e = order[k];
        int64_t bg = LLONG_MAX;
        int32_t bp = INT32_MAX;
        for (int p = lane; p < P; p += kWave) {
            if (nfill[p] < H && (G[p] < bg || (G[p] == bg && p < bp))) {
                bg = G[p];
                bp = p;
            }
        }
#pragma unroll
        for (int d = 32; d >= 1; d >>= 1) {
            const int64_t og = __shfl_xor(bg, d, kWave);
            const int32_t op = __shfl_xor(bp, d, kWave);
            if (og < bg || (og == bg && op < bp)) {
                bg = og;
                bp = op;
            }
        }
        if (lane == 0) {
            const int32_t v = bp * H + nfill[bp];
            slot_of[(int64_t)l * E + e] = v;
            if (expert_at_slot) expert_at_slot[(int64_t)l * E + v] = e;
            G[bp] += Ll[e];
            nfill[bp] += 1;
        }
        __syncthreads();
    }
    for (int p = lane; p < P; p += kWave) rank_load[(int64_t)l * P + p] = G[p];
}

// q[i][l][p] = sum_{h<H} demand[i][l][expert_at_slot[l][p*H + h]].  A
// workgroup owns one layer and a tile of samples: it stages the tile's
// demand rows (contiguous E-int32 rows, coalesced) in LDS and gathers each
// rank's H experts from there.
__global__ void __launch_bounds__(256) k_project(const int32_t *__restrict__ demand,
                                                 const int32_t *__restrict__ expert_at_slot,
                                                 int32_t *__restrict__ q, int32_t N, int32_t L,
                                                 int32_t E, int32_t P, int32_t tile) {
    extern __shared__ char smem[];
    int32_t *eas = reinterpret_cast<int32_t *>(smem);  // [E]
    int32_t *rows = eas + E;                             // [tile][E]
    const int l = blockIdx.x;
    const int32_t H = E / P;
    for (int v = threadIdx.x; v < E; v += blockDim.x) eas[v] = expert_at_slot[(int64_t)l * E + v];
    const int64_t i0 = (int64_t)blockIdx.y * tile;
    int32_t ns = tile;
    if (i0 + ns > N) ns = (int32_t)(N - i0);
    for (int64_t x = threadIdx.x; x < (int64_t)ns * E; x += blockDim.x) {
        const int64_t s = x / E, e = x % E;
        rows[x] = demand[((i0 + s) * L + l) * E + e];
    }
    __syncthreads();
    for (int64_t x = threadIdx.x; x < (int64_t)ns * P; x += blockDim.x) {
        const int64_t s = x / P, p = x % P;
        const int32_t *row = rows + s * E;
        int32_t acc = 0;
        for (int h = 0; h < H; ++h) acc += row[eas[p * H + h]];
        q[((i0 + s) * L + l) * P + p] = acc;
    }
}

// A given placement pi_l: checks that it is a permutation of the E slots (an
// LDS inverse filled by compare-and-swap: no slot out of range and no slot
// taken twice), writes the inverse for k_project and sums every rank's
// aggregate (Eq. placement-load).  One workgroup per layer.
__global__ void __launch_bounds__(256) k_given_place(const int64_t *__restrict__ agg,
                                                     const int32_t *__restrict__ slot_of, int32_t E,
                                                     int32_t P, int32_t *__restrict__ expert_at_slot,
                                                     int64_t *__restrict__ rank_load, int32_t *bad) {
    extern __shared__ char smem[];
    int32_t *eas = reinterpret_cast<int32_t *>(smem);  // [E]
    const int l = blockIdx.x;
    for (int v = threadIdx.x; v < E; v += blockDim.x) eas[v] = -1;
    __syncthreads();
    bool ok = true;
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
        const int32_t v = slot_of[(int64_t)l * E + e];
        if (v < 0 || v >= E || atomicCAS(&eas[v], -1, e) != -1) ok = false;
    }
    if (!ok) atomicOr(bad, 1);
    __syncthreads();
    for (int v = threadIdx.x; v < E; v += blockDim.x) expert_at_slot[(int64_t)l * E + v] = eas[v];
    const int32_t H = E / P;
    for (int p = threadIdx.x; p < P; p += blockDim.x) {
        int64_t sum = 0;
        for (int h = 0; h < H; ++h) {
            const int32_t e = eas[p * H + h];
            sum += e >= 0 ? agg[(int64_t)l * E + e] : 0;
        }
        rank_load[(int64_t)l * P + p] = sum;
    }
}

}  // namespace rp

using namespace rp;

namespace {

int launch_project(const int32_t *demand, const int32_t *eas, int32_t *q, int32_t N, int32_t L, int32_t E,
                   int32_t P, hipStream_t stream) {
    int32_t tile = 8192 / E;
    if (tile < 1) tile = 1;
    if (tile > 64) tile = 64;
    const size_t lds2 = (size_t)E * 4 + (size_t)tile * E * 4;
    if (lds2 > 160 * 1024) return ROUTEPACK_E_UNSUPPORTED;
    const unsigned gy = (unsigned)((N + tile - 1) / tile);
    hipLaunchKernelGGL(k_project, dim3(L, gy), dim3(256), lds2, stream, demand, eas, q, N, L, E, P, tile);
    return ROUTEPACK_OK;
}

}  // namespace

extern "C" int routepack_aggregate_demand(const routepack_problem *prob, const int32_t *demand,
                                          int64_t *agg, hipStream_t stream) {
    if (!prob || !agg || (!demand && prob->n_samples > 0)) return ROUTEPACK_E_INVALID;
    if (prob->n_samples < 0 || prob->n_layers < 0 || prob->n_experts < 1) return ROUTEPACK_E_INVALID;
    const int64_t N = prob->n_samples, M = (int64_t)prob->n_layers * prob->n_experts;
    if (M == 0) return ROUTEPACK_OK;
    hipLaunchKernelGGL(k_fill_i64, dim3((unsigned)((M + 255) / 256 < 1024 ? (M + 255) / 256 : 1024)),
                       dim3(256), 0, stream, agg, M, (int64_t)0);
    if (N > 0) {
        const bool vec = (M % 4 == 0) && ((uintptr_t)demand % 16 == 0);
        const int64_t cols_per_block = 256 * (vec ? 4 : 1);
        const int64_t gx = (M + cols_per_block - 1) / cols_per_block;
        int64_t gy = 8192 / gx;
        if (gy < 1) gy = 1;
        if (gy > N) gy = N;
        if (gy > 65535) gy = 65535;
        const int64_t band = (N + gy - 1) / gy;
        gy = (N + band - 1) / band;
        if (vec)
            hipLaunchKernelGGL(k_aggregate<4>, dim3((unsigned)gx, (unsigned)gy), dim3(256), 0,
                               stream, demand, agg, N, M, band);
        else
            hipLaunchKernelGGL(k_aggregate<1>, dim3((unsigned)gx, (unsigned)gy), dim3(256), 0,
                               stream, demand, agg, N, M, band);
    }
    return hipGetLastError() == hipSuccess ? ROUTEPACK_OK : ROUTEPACK_E_DEVICE;
}

extern "C" int routepack_place_experts(const routepack_problem *prob, const int64_t *agg,
                                       int32_t *slot_of, int64_t *rank_load,
                                       const int32_t *demand, int32_t *q, hipStream_t stream) {
    if (!prob || !agg || !slot_of || !rank_load) return ROUTEPACK_E_INVALID;
    const int32_t L = prob->n_layers, E = prob->n_experts, P = prob->n_ranks, N = prob->n_samples;
    if (L < 0 || E < 1 || P < 1 || E % P != 0 || N < 0) return ROUTEPACK_E_INVALID;
    if (L == 0) return ROUTEPACK_OK;
    const bool want_q = demand && q && N > 0;
    Scratch scr(stream);
    int32_t *eas = want_q ? scr.get<int32_t>((size_t)L * E) : nullptr;
    if (scr.failed()) return ROUTEPACK_E_DEVICE;
    const size_t lds = (size_t)E * 8 + (size_t)P * 8 + (size_t)E * 4 + (size_t)P * 4;
    if (lds > 160 * 1024) return ROUTEPACK_E_UNSUPPORTED;
    hipLaunchKernelGGL(k_lpt_place, dim3(L), dim3(64), lds, stream, agg, E, P, slot_of, rank_load,
                       eas);
    if (want_q) RP_TRY(launch_project(demand, eas, q, N, L, E, P, stream));
    return hipGetLastError() == hipSuccess ? ROUTEPACK_OK : ROUTEPACK_E_DEVICE;
}

extern "C" int routepack_project_demand(const routepack_problem *prob, const int64_t *agg,
                                        const int32_t *slot_of, int64_t *rank_load, const int32_t *demand,
                                        int32_t *q, hipStream_t stream) {
    if (!prob || !agg || !slot_of || !rank_load) return ROUTEPACK_E_INVALID;
    const int32_t L = prob->n_layers, E = prob->n_experts, P = prob->n_ranks, N = prob->n_samples;
    if (L < 0 || E < 1 || P < 1 || E % P != 0 || N < 0) return ROUTEPACK_E_INVALID;
    if (L == 0) return ROUTEPACK_OK;
    if ((size_t)E * 4 > 160 * 1024) return ROUTEPACK_E_UNSUPPORTED;
    Scratch scr(stream);
    int32_t *eas = scr.get<int32_t>((size_t)L * E);
    int32_t *bad = scr.get<int32_t>(1);
    if (scr.failed()) return ROUTEPACK_E_DEVICE;
    RP_HIP(hipMemsetAsync(bad, 0, sizeof(int32_t), stream));
    hipLaunchKernelGGL(k_given_place, dim3(L), dim3(256), (size_t)E * 4, stream, agg, slot_of, E, P, eas,
                       rank_load, bad);
    RP_HIP(hipGetLastError());
    int32_t h_bad = 0;
    RP_HIP(hipMemcpyAsync(&h_bad, bad, sizeof(h_bad), hipMemcpyDeviceToHost, stream));
    RP_HIP(hipStreamSynchronize(stream));
    if (h_bad) return ROUTEPACK_E_INVALID;
    if (demand && q && N > 0) RP_TRY(launch_project(demand, eas, q, N, L, E, P, stream));
    return hipGetLastError() == hipSuccess ? ROUTEPACK_OK : ROUTEPACK_E_DEVICE;
}
