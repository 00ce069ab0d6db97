// Window demand aggregation (Sec. 3.3), layer-local LPT placement (Alg. 1)
// and the physical-rank projection (Eq. physical-rank-demand) on gfx950.
//
// Aggregation is an HBM stream: the [N][L*E] int32 demand matrix is reduced
// over its rows in two passes and without atomics.  A workgroup owns 256
// columns (4 per lane: one 16-byte load per row, 1 KiB contiguous per wave)
// and a band of at least 64 rows; its four waves take every fourth row with
// eight loads in flight each, sum in int64 registers, meet in LDS and write
// one int64 partial per column and band.  A second kernel sums the bands of
// each column (the partials are at most 2/64 of the bytes read).  Integer
// sums are exact, so the result does not depend on the order.
#include <mutex>
#include <optional>
#include <type_traits>

#include "rp_device.h"
#include "rp_internal.h"

namespace rp {

// Band partials of routepack_aggregate_demand_noalloc: a fixed device array
// (each device the library runs on holds its own copy until the process
// ends).  In host code `scratch` is only a stand-in for the symbol: its
// device address comes from hipGetSymbolAddress, once per device.
constexpr int64_t kAggScratchElems = (int64_t)1 << 20;  // 8 MiB of int64 partials
static __device__ __align__(256) int64_t scratch[kAggScratchElems];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
int64_t *g_scratch_ptr[kMaxDevices];

// The current device's address of `scratch` (looked up on the first call on
// that device, with it current); nullptr on a HIP error.
int64_t *agg_scratch_on_current_device() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
        g_scratch_ptr[dev] = static_cast<int64_t *>(ptr);
    }
    return g_scratch_ptr[dev];
}
}  // namespace

__global__ void k_fill_i64(int64_t *p, int64_t n, int64_t v) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

template <int VEC>
__global__ void __launch_bounds__(256) k_aggregate_bands(const int32_t *__restrict__ demand,
                                                         int64_t *__restrict__ part, int32_t n_rows,
                                                         int64_t n_cols, int32_t band) {
    __shared__ int64_t red[3][64 * VEC];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int64_t col = ((int64_t)blockIdx.x * 64 + lane) * VEC;
    const int32_t r0 = (int32_t)blockIdx.y * band;
    const int32_t r1 = r0 + band < n_rows ? r0 + band : n_rows;
    int64_t acc[VEC];
#pragma unroll
    for (int c = 0; c < VEC; ++c) acc[c] = 0;
    if (col < n_cols) {
        // the host takes VEC = 4 only when n_cols % 4 == 0 and rows are 16-byte aligned
        const int32_t *p = demand + (int64_t)(r0 + wv) * n_cols + col;
        const int64_t step = 4 * n_cols;
        int32_t r = r0 + wv;
        if (VEC == 4) {
            for (; r + 28 < r1; r += 32) {
                int4 v[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) v[u] = *reinterpret_cast<const int4 *>(p + u * step);
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    acc[0] += v[u].x;
                    acc[1 % VEC] += v[u].y;
                    acc[2 % VEC] += v[u].z;
                    acc[3 % VEC] += v[u].w;
                }
                p += 8 * step;
            }
            for (; r < r1; r += 4) {
                const int4 a = *reinterpret_cast<const int4 *>(p);
                acc[0] += a.x;
                acc[1 % VEC] += a.y;
                acc[2 % VEC] += a.z;
                acc[3 % VEC] += a.w;
                p += step;
            }
        } else {
            for (; r < r1; r += 4) {
                acc[0] += *p;
                p += step;
            }
        }
    }
    if (wv > 0)
#pragma unroll
        for (int c = 0; c < VEC; ++c) red[wv - 1][lane * VEC + c] = acc[c];
    __syncthreads();
    if (wv == 0 && col < n_cols) {
        int64_t *dst = part + (int64_t)blockIdx.y * n_cols + col;
#pragma unroll
        for (int c = 0; c < VEC; ++c)
            dst[c] = acc[c] + red[0][lane * VEC + c] + red[1][lane * VEC + c] + red[2][lane * VEC + c];
    }
}

// agg[c] = sum over the bands of part[b][c]: a workgroup owns 64 columns,
// its four waves take every fourth band and meet in LDS.
__global__ void __launch_bounds__(256) k_aggregate_cols(const int64_t *__restrict__ part, int32_t n_bands,
                                                        int64_t n_cols, int64_t *__restrict__ agg) {
    __shared__ int64_t red[3][64];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int64_t col = (int64_t)blockIdx.x * 64 + lane;
    int64_t s0 = 0, s1 = 0;
    if (col < n_cols) {
        int32_t b = wv;
        for (; b + 4 < n_bands; b += 8) {
            s0 += part[(int64_t)b * n_cols + col];
            s1 += part[(int64_t)(b + 4) * n_cols + col];
        }
        for (; b < n_bands; b += 4) s0 += part[(int64_t)b * n_cols + col];
    }
    s0 += s1;
    if (wv > 0) red[wv - 1][lane] = s0;
    __syncthreads();
    if (wv == 0 && col < n_cols) agg[col] = s0 + red[0][lane] + red[1][lane] + red[2][lane];
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
    if (P <= kWave) {
        // lane p holds rank p's load and fill; a step is a wave minimum of
        // the loads of ranks with room, then the lowest such lane (the
        // order of the next 64 experts is held one per lane)
        int64_t g = 0;
        int32_t nf = 0, oe = 0;
        int64_t ol = 0;
        for (int k = 0; k < E; ++k) {
            if ((k & (kWave - 1)) == 0) {
                oe = k + lane < E ? order[k + lane] : 0;
                ol = Ll[oe];
            }
            const int e = __builtin_amdgcn_readlane(oe, k & (kWave - 1));
            const int64_t le = (int64_t)readlane64((uint64_t)ol, k & (kWave - 1));
            const bool avail = lane < P && nf < H;
            const int64_t mn = wave_min(avail ? g : LLONG_MAX);
            const int bp = first_lane(__ballot(avail && g == mn));
            if (lane == bp) {
                const int32_t v = bp * H + nf;
                slot_of[(int64_t)l * E + e] = v;
                if (expert_at_slot) expert_at_slot[(int64_t)l * E + v] = e;
                g += le;
                ++nf;
            }
        }
        if (lane < P) rank_load[(int64_t)l * P + lane] = g;
        return;
    }
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
template <bool V4, int HC>
__global__ void __launch_bounds__(256) k_project(const int32_t *__restrict__ demand,
                                                 const int32_t *__restrict__ expert_at_slot,
                                                 int32_t *__restrict__ q, int32_t N, int32_t L,
                                                 int32_t E, int32_t P, int32_t tile) {
    using Word = typename std::conditional<V4, int4, int32_t>::type;
    extern __shared__ __align__(16) char smem[];
    int32_t *rows = reinterpret_cast<int32_t *>(smem);  // [tile][E]
    int32_t *eas = rows + (int64_t)tile * E;             // [E]
    const int l = blockIdx.x, tid = threadIdx.x, nt = blockDim.x;
    const int32_t H = E / P;
    for (int v = tid; v < E; v += nt) eas[v] = expert_at_slot[(int64_t)l * E + v];
    const int32_t i0 = (int32_t)blockIdx.y * tile;
    const int32_t ns = tile < N - i0 ? tile : N - i0;
    const int64_t stride = (int64_t)L * E;  // between consecutive samples' rows
    const int32_t *src = demand + ((int64_t)i0 * L + l) * E;
    // Stage the tile's rows: threads split into groups of one row's width
    // (in 16-byte words when E % 4 == 0 and the rows are 16-byte aligned),
    // a group per sample at a time.
    const int32_t width = V4 ? E >> 2 : E;
    const int32_t per = width < nt ? nt / width : 1;  // samples per pass
    const int32_t s0 = width < nt ? tid / width : 0;
    const int32_t x0 = width < nt ? tid - s0 * width : tid;
    const Word *srcw = reinterpret_cast<const Word *>(src);
    Word *rowsw = reinterpret_cast<Word *>(rows);
    const int64_t sw = V4 ? stride >> 2 : stride;  // the strides in words
    if (width < nt && s0 < per) {
        // U rows per thread: every load issued before the first store (the
        // rows past the tile repeat its last row and are not stored)
        constexpr int U = 8;
        for (int32_t s = s0; s < ns; s += U * per) {
            Word v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t su = s + u * per < ns ? s + u * per : ns - 1;
                v[u] = srcw[(int64_t)su * sw + x0];
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
                if (s + u * per < ns) rowsw[(int64_t)(s + u * per) * width + x0] = v[u];
        }
    } else if (width >= nt) {
        for (int32_t s = 0; s < ns; ++s)
            for (int32_t x = tid; x < width; x += nt) rowsw[(int64_t)s * width + x] = srcw[(int64_t)s * sw + x];
    }
    __syncthreads();
    // q[i0 + s][l][p] = the sum of the tile row s over rank p's H slots; a
    // thread keeps its rank's H experts in registers when H == HC
    const int32_t perq = P < nt ? nt / P : 1;
    const int32_t sq = P < nt ? tid / P : 0;
    const int32_t p0 = P < nt ? tid - sq * P : tid;
    if (sq < perq) {
        for (int32_t p = p0; p < P; p += (P < nt ? P : nt)) {
            if (HC > 0) {
                int32_t ex[HC > 0 ? HC : 1];
#pragma unroll
                for (int h = 0; h < HC; ++h) ex[h] = eas[p * HC + h];
                for (int32_t s = sq; s < ns; s += perq) {
                    const int32_t *row = rows + (int64_t)s * E;
                    int32_t acc = 0;
#pragma unroll
                    for (int h = 0; h < HC; ++h) acc += row[ex[h]];
                    q[((int64_t)(i0 + s) * L + l) * P + p] = acc;
                }
            } else {
                for (int32_t s = sq; s < ns; s += perq) {
                    const int32_t *row = rows + (int64_t)s * E;
                    int32_t acc = 0;
                    for (int h = 0; h < H; ++h) acc += row[eas[p * H + h]];
                    q[((int64_t)(i0 + s) * L + l) * P + p] = acc;
                }
            }
        }
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
    const size_t lds2 = (size_t)tile * E * 4 + (size_t)E * 4;
    if (lds2 > 160 * 1024) return ROUTEPACK_E_UNSUPPORTED;
    const bool v4 = (E % 4 == 0) && ((uintptr_t)demand % 16 == 0);
    const int32_t H = E / P;
    const unsigned gy = (unsigned)((N + tile - 1) / tile);
    auto go = [&](auto kern) -> int {
        if (lds2 > 64 * 1024 &&
            hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds2) !=
                hipSuccess)
            return ROUTEPACK_E_DEVICE;
        hipLaunchKernelGGL(kern, dim3(L, gy), dim3(256), lds2, stream, demand, eas, q, N, L, E, P, tile);
        return ROUTEPACK_OK;
    };
    if (v4) {
        switch (H) {
            case 4: return go(k_project<true, 4>);
            case 8: return go(k_project<true, 8>);
            case 16: return go(k_project<true, 16>);
            default: return go(k_project<true, 0>);
        }
    }
    return go(k_project<false, 0>);
}

}  // namespace

// Both aggregation entry points: the band grid, then the two passes.  With
// max_part > 0 the partials go to `fixed` (at most max_part int64 entries,
// fewer bands when needed) instead of stream-ordered scratch.
static int aggregate_demand(const routepack_problem *prob, const int32_t *demand, int64_t *agg,
                            int64_t *fixed, int64_t max_part, hipStream_t stream) {
    if (!prob || !agg || (!demand && prob->n_samples > 0)) return ROUTEPACK_E_INVALID;
    if (prob->n_samples < 0 || prob->n_layers < 0 || prob->n_experts < 1) return ROUTEPACK_E_INVALID;
    const int64_t N = prob->n_samples, M = (int64_t)prob->n_layers * prob->n_experts;
    if (max_part > 0 && M > max_part) return ROUTEPACK_E_UNSUPPORTED;  // not even one band fits
    if (M == 0) return ROUTEPACK_OK;
    if (N == 0) {
        hipLaunchKernelGGL(k_fill_i64, dim3((unsigned)((M + 255) / 256 < 1024 ? (M + 255) / 256 : 1024)),
                           dim3(256), 0, stream, agg, M, (int64_t)0);
        return hipGetLastError() == hipSuccess ? ROUTEPACK_OK : ROUTEPACK_E_DEVICE;
    }
    const bool vec = (M % 4 == 0) && ((uintptr_t)demand % 16 == 0);
    const int64_t gx = (M + 64 * (vec ? 4 : 1) - 1) / (64 * (vec ? 4 : 1));
    // about 4096 workgroups, but bands of at least 64 rows
    int64_t gy = (4096 + gx - 1) / gx, cap = N / 64 > 1 ? N / 64 : 1;
    if (gy > cap) gy = cap;
    if (gy > 65535) gy = 65535;
    if (max_part > 0 && gy * M > max_part) gy = max_part / M;  // >= 1 (checked above)
    const int32_t band = (int32_t)((N + gy - 1) / gy);
    gy = (N + band - 1) / band;
    if (gx > 2147483647LL) return ROUTEPACK_E_UNSUPPORTED;
    std::optional<Scratch> scr;  // (none with a fixed partials buffer)
    int64_t *part = fixed;
    if (!part) {
        scr.emplace(stream);
        part = scr->get<int64_t>((size_t)gy * M);
        if (scr->failed()) return ROUTEPACK_E_DEVICE;
    }
    if (vec)
        hipLaunchKernelGGL(k_aggregate_bands<4>, dim3((unsigned)gx, (unsigned)gy), dim3(256), 0, stream, demand,
                           part, (int32_t)N, M, band);
    else
        hipLaunchKernelGGL(k_aggregate_bands<1>, dim3((unsigned)gx, (unsigned)gy), dim3(256), 0, stream, demand,
                           part, (int32_t)N, M, band);
    hipLaunchKernelGGL(k_aggregate_cols, dim3((unsigned)((M + 63) / 64)), dim3(256), 0, stream,
                       (const int64_t *)part, (int32_t)gy, M, agg);
    return hipGetLastError() == hipSuccess ? ROUTEPACK_OK : ROUTEPACK_E_DEVICE;
}

extern "C" int routepack_aggregate_demand(const routepack_problem *prob, const int32_t *demand,
                                          int64_t *agg, hipStream_t stream) {
    return aggregate_demand(prob, demand, agg, nullptr, 0, stream);
}

extern "C" int routepack_aggregate_demand_noalloc(const routepack_problem *prob, const int32_t *demand,
                                                  int64_t *agg, hipStream_t stream) {
    if (!prob || !agg || (!demand && prob->n_samples > 0)) return ROUTEPACK_E_INVALID;
    if (prob->n_layers < 0 || prob->n_experts < 1) return ROUTEPACK_E_INVALID;
    if ((int64_t)prob->n_layers * prob->n_experts > kAggScratchElems) return ROUTEPACK_E_UNSUPPORTED;
    int64_t *part = agg_scratch_on_current_device();
    if (!part) return ROUTEPACK_E_DEVICE;
    return aggregate_demand(prob, demand, agg, part, kAggScratchElems, stream);
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
