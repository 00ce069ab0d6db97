// Lower bound on the row count of a fixed-row layout (arXiv 2608.12146,
// Sec. 3.2, Eqs. token-capacity and min-row-count): R* is minimal when a
// valid lower bound on the number of capacity-C cells reaches R* D.  Beside
// the token volume, this takes the cardinality bounds (no cell holds k + 1
// samples longer than C / (k + 1)) and Martello and Toth's L2 (Discrete
// Applied Mathematics 28, 1990), each a count or a sum over a threshold of
// the lengths sorted in decreasing order:
//   k_sorted_lengths  the lengths in (-t, i) order, as int64
//   k_prefix          their exclusive prefix sums (one workgroup)
//   k_cell_bounds     thread u evaluates the cardinality bound for k = u + 1
//                     and L2 at alpha = the u-th length when it is at most
//                     C / 2 (thread 0 also alpha = 0 and the volume); the
//                     largest goes to one atomic maximum.
// And the fixed-bin feasibility check itself (Eq. min-row-count: is the
// feasible set X_R non-empty?) as a depth-first branch and bound under a
// node budget, in a fixed order so that its verdict, node count and first
// solution are defined:
//   k_fixed_bin       one wave, the cell loads and the choices in LDS, the
//                     sorted lengths read from memory: samples in (-t, i) order go to an open cell
//                     with room, lowest index first (a 64-lane ballot per
//                     64 cells), then to the first unopened cell; a sample
//                     equal in length to the previous one goes to no lower
//                     cell; a branch is cut when fewer samples remain than
//                     unopened cells.  Every iteration places a sample
//                     (counted against the budget) or undoes one, so the
//                     loop ends within twice the budget plus N iterations.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "routepack.h"
#include "rp_device.h"
#include "rp_internal.h"

namespace rp {
namespace {

__global__ void k_sorted_lengths(const int32_t *t, const int32_t *sigma, int32_t N, int64_t *ts) {
    const int32_t u = blockIdx.x * blockDim.x + threadIdx.x;
    if (u < N) ts[u] = t[sigma[u]];
}

// ps[u] = sum_{v < u} ts[v] for u in [0, N]; one workgroup of 1024 threads,
// each summing a contiguous chunk.
__global__ void __launch_bounds__(1024) k_prefix(const int64_t *ts, int32_t N, int64_t *ps) {
    __shared__ int64_t part[1024];
    const int tid = threadIdx.x;
    const int32_t per = (N + 1023) / 1024, lo = tid * per < N ? tid * per : N, hi = lo + per < N ? lo + per : N;
    int64_t sum = 0;
    for (int32_t u = lo; u < hi; ++u) sum += ts[u];
    part[tid] = sum;
    __syncthreads();
    if (tid == 0) {
        int64_t run = 0;
        for (int w = 0; w < 1024; ++w) {
            const int64_t v = part[w];
            part[w] = run;
            run += v;
        }
        ps[N] = run;
    }
    __syncthreads();
    int64_t run = part[tid];
    for (int32_t u = lo; u < hi; ++u) {
        ps[u] = run;
        run += ts[u];
    }
}

// ts[u] = t[sigma[u]] as int32: the lengths in (-t, i) order for the search.
__global__ void k_sorted_lengths32(const int32_t *t, const int32_t *sigma, int32_t N, int32_t *ts) {
    const int32_t u = blockIdx.x * blockDim.x + threadIdx.x;
    if (u < N) ts[u] = t[sigma[u]];
}

// #{u : ts[u] > x} in the decreasing array ts.
__device__ inline int32_t count_above(const int64_t *ts, int32_t N, int64_t x) {
    int32_t lo = 0, hi = N;  // ts[< lo] > x, ts[>= hi] <= x
    while (lo < hi) {
        const int32_t md = lo + ((hi - lo) >> 1);
        if (ts[md] > x) lo = md + 1;
        else hi = md;
    }
    return lo;
}

__device__ inline int64_t ceil_div(int64_t a, int64_t b) { return a >= 0 ? (a + b - 1) / b : -((-a) / b); }

// L2 of Martello and Toth at threshold alpha (0 <= alpha <= C/2).
__device__ inline int64_t l2_at(const int64_t *ts, const int64_t *ps, int32_t N, int64_t C, int64_t alpha) {
    const int32_t j1 = count_above(ts, N, C - alpha);   // t > C - alpha
    const int32_t b = count_above(ts, N, C / 2);        // t > C/2
    const int32_t e = count_above(ts, N, alpha - 1);    // t >= alpha
    const int64_t n2 = b - j1, s2 = ps[b] - ps[j1], s3 = ps[e] - ps[b];
    const int64_t extra = ceil_div(s3 - (n2 * C - s2), C);
    return (int64_t)j1 + n2 + (extra > 0 ? extra : 0);
}

__global__ void k_cell_bounds(const int64_t *ts, const int64_t *ps, int32_t N, int64_t C,
                              unsigned long long *best) {
    const int32_t u = blockIdx.x * blockDim.x + threadIdx.x;
    if (u >= N) return;
    const int64_t k = (int64_t)u + 1;
    int64_t v = ceil_div(count_above(ts, N, C / (k + 1)), k);  // (k + 1) t > C
    if (2 * ts[u] <= C) {
        const int64_t l = l2_at(ts, ps, N, C, ts[u]);
        v = l > v ? l : v;
    }
    if (u == 0) {
        const int64_t l = l2_at(ts, ps, N, C, 0), vol = ceil_div(ps[N], C);
        v = l > v ? l : v;
        v = vol > v ? vol : v;
    }
    atomicMax(best, (unsigned long long)v);
}

__global__ void __launch_bounds__(kWave) k_fixed_bin(const int32_t *__restrict__ ts, int32_t n, int64_t C,
                                                     int32_t K, int64_t budget, const int32_t *__restrict__ sigma,
                                                     int64_t *out, int32_t *cells) {
    extern __shared__ __align__(16) char smem[];
    int64_t *load = reinterpret_cast<int64_t *>(smem);       // [K]
    int32_t *choice = reinterpret_cast<int32_t *>(load + K);  // [n] cell of sample h, -1 none
    const int lane = lane_id();
    for (int32_t c = lane; c < K; c += kWave) load[c] = 0;
    for (int32_t u = lane; u < n; u += kWave) choice[u] = -1;
    __syncthreads();
    int32_t h = 0, opened = 0;
    int64_t nodes = 0, status = 0;
    for (;;) {
        if (h == n) {  // every sample placed; the cut leaves no cell unopened
            status = 1;
            break;
        }
        const int64_t th = ts[h];
        const int32_t ch = choice[h];
        int32_t lo = ch + 1;
        if (ch < 0 && h > 0 && th == ts[h - 1]) lo = choice[h - 1];
        int32_t b = -1;
        for (int32_t base = lo; base < opened && b < 0; base += kWave) {
            const int32_t c = base + lane;
            const uint64_t fit = __ballot(c < opened && load[c] + th <= C);
            if (fit) b = base + first_lane(fit);
        }
        if (b < 0 && lo <= opened && opened < K) b = opened;
        if (b >= 0) {
            if (nodes == budget) {  // the next placement would exceed the budget
                status = 2;
                break;
            }
            ++nodes;
            const bool fresh = b == opened;
            opened += fresh ? 1 : 0;
            if (lane == 0) {
                load[b] += th;
                choice[h] = b;
            }
            __syncthreads();
            if (n - (h + 1) >= K - opened) {
                ++h;
                continue;  // (choice[h] is -1: set at the start, reset when left)
            }
            if (lane == 0) load[b] -= th;  // cut: undo, then the next cell for h
            __syncthreads();
            opened -= fresh ? 1 : 0;
            continue;
        }
        // backtrack: sample h has no cell left
        if (lane == 0) choice[h] = -1;
        __syncthreads();
        if (--h < 0) {
            status = 0;
            break;
        }
        const int32_t pb = choice[h];
        if (lane == 0) load[pb] -= ts[h];
        __syncthreads();
        if (load[pb] == 0) --opened;  // it was the last cell opened
    }
    if (lane == 0) {
        out[0] = status;
        out[1] = nodes;
    }
    if (status == 1 && cells)
        for (int32_t u = lane; u < n; u += kWave) cells[sigma[u]] = choice[u];
}

}  // namespace
}  // namespace rp

using namespace rp;

extern "C" int routepack_row_lower_bound(const routepack_problem *prob, const int32_t *lengths, int32_t *r_bound,
                                         int64_t *cell_bound, hipStream_t stream) {
    Topology topo;
    RP_TRY(check_problem(prob, &topo));
    if (!lengths || !r_bound) return ROUTEPACK_E_INVALID;
    const int32_t N = prob->n_samples;
    const int64_t C = prob->capacity;
    WindowStats ws;
    RP_TRY(window_stats(prob, lengths, nullptr, &ws, stream));
    if (ws.min_t < 1 || ws.max_t > C) return ROUTEPACK_E_INFEASIBLE;
    Scratch scr(stream);
    int32_t *sigma = scr.get<int32_t>(N);
    int64_t *ts = scr.get<int64_t>(N);
    int64_t *ps = scr.get<int64_t>((size_t)N + 1);
    unsigned long long *best = scr.get<unsigned long long>(1);
    if (scr.failed()) return ROUTEPACK_E_DEVICE;
    RP_HIP(hipMemsetAsync(best, 0, sizeof(*best), stream));
    RP_TRY(rank_sort_desc(lengths, N, sigma, stream));
    hipLaunchKernelGGL(k_sorted_lengths, dim3((N + 255) / 256), dim3(256), 0, stream, lengths, sigma, N, ts);
    hipLaunchKernelGGL(k_prefix, dim3(1), dim3(1024), 0, stream, (const int64_t *)ts, N, ps);
    hipLaunchKernelGGL(k_cell_bounds, dim3((N + 255) / 256), dim3(256), 0, stream, (const int64_t *)ts,
                       (const int64_t *)ps, N, C, best);
    RP_HIP(hipGetLastError());
    unsigned long long k = 0;
    RP_HIP(hipMemcpyAsync(&k, best, sizeof(k), hipMemcpyDeviceToHost, stream));
    RP_HIP(hipStreamSynchronize(stream));
    const int64_t D = topo.D;
    int64_t r = ((int64_t)k + D - 1) / D;
    if (r < 1) r = 1;
    if (prob->min_rows > r) r = prob->min_rows;
    *r_bound = (int32_t)r;
    if (cell_bound) *cell_bound = (int64_t)k;
    return ROUTEPACK_OK;
}

extern "C" int routepack_fixed_bin_search(const routepack_problem *prob, const int32_t *lengths, int32_t n_rows,
                                          int64_t node_budget, int32_t *status, int64_t *nodes, int32_t *layout,
                                          hipStream_t stream) {
    Topology topo;
    RP_TRY(check_problem(prob, &topo));
    if (!lengths || !status || n_rows < 1 || node_budget < 0) return ROUTEPACK_E_INVALID;
    const int32_t N = prob->n_samples;
    const int64_t C = prob->capacity, K64 = (int64_t)n_rows * topo.D;
    WindowStats ws;
    RP_TRY(window_stats(prob, lengths, nullptr, &ws, stream));
    if (ws.min_t < 1) return ROUTEPACK_E_INVALID;
    if (K64 > N || ws.max_t > C) {  // no layout: more cells than samples, or a sample over capacity
        *status = 0;
        if (nodes) *nodes = 0;
        return ROUTEPACK_OK;
    }
    const int32_t K = (int32_t)K64;
    const size_t lds = 8 * (size_t)K + 4 * (size_t)N;
    if (lds > 150 * 1024) return ROUTEPACK_E_UNSUPPORTED;
    Scratch scr(stream);
    int32_t *sigma = scr.get<int32_t>(N);
    int32_t *ts = scr.get<int32_t>(N);
    int64_t *out = scr.get<int64_t>(2);
    if (scr.failed()) return ROUTEPACK_E_DEVICE;
    RP_TRY(rank_sort_desc(lengths, N, sigma, stream));
    hipLaunchKernelGGL(k_sorted_lengths32, dim3((N + 255) / 256), dim3(256), 0, stream, lengths,
                       (const int32_t *)sigma, N, ts);
    if (hipFuncSetAttribute((const void *)k_fixed_bin, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
        hipSuccess)
        return ROUTEPACK_E_DEVICE;
    hipLaunchKernelGGL(k_fixed_bin, dim3(1), dim3(kWave), lds, stream, (const int32_t *)ts, N, C, K, node_budget,
                       (const int32_t *)sigma, out, layout);
    RP_HIP(hipGetLastError());
    int64_t h[2] = {0, 0};
    RP_HIP(hipMemcpyAsync(h, out, sizeof(h), hipMemcpyDeviceToHost, stream));
    RP_HIP(hipStreamSynchronize(stream));
    *status = (int32_t)h[0];
    if (nodes) *nodes = h[1];
    return ROUTEPACK_OK;
}
