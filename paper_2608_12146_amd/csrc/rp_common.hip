// Validation, scratch, window bounds and status strings for the RoutePack
// C-ABI library.
#include <atomic>
#include <map>
#include <math.h>
#include <mutex>
#include <string.h>
#include <thread>
#include <utility>

#include "rp_device.h"
#include "rp_internal.h"

namespace rp {

int check_problem(const routepack_problem *p, Topology *topo) {
    if (!p) return ROUTEPACK_E_INVALID;
    if (p->n_samples < 1 || p->n_layers < 0 || p->n_experts < 1 || p->n_ranks < 1)
        return ROUTEPACK_E_INVALID;
    if (p->n_experts % p->n_ranks != 0) return ROUTEPACK_E_INVALID;
    if (p->n_dp < 1 || p->n_edp < 1 || p->n_edp > p->n_dp) return ROUTEPACK_E_INVALID;
    if (p->capacity < 1 || p->n_stages < 1 || p->frac_bits < 0 || p->frac_bits > 30)
        return ROUTEPACK_E_INVALID;
    if (p->min_rows < 1 || !p->dp_to_edp || !p->alpha_fp || !p->beta_fp) return ROUTEPACK_E_INVALID;
    for (int s = 0; s < p->n_stages; ++s)
        if (p->alpha_fp[s] < 0 || p->beta_fp[s] < 0) return ROUTEPACK_E_INVALID;
    Topology t;
    t.D = p->n_dp;
    t.G = p->n_edp;
    t.count.assign(t.G, 0);
    t.slots.assign((size_t)t.G * t.D, 0);
    for (int d = 0; d < t.D; ++d) {
        const int g = p->dp_to_edp[d];
        if (g < 0 || g >= t.G) return ROUTEPACK_E_INVALID;
        t.slots[(size_t)g * t.D + t.count[g]++] = d;
    }
    for (int g = 0; g < t.G; ++g) {
        if (t.count[g] == 0) return ROUTEPACK_E_INVALID;
        if (t.count[g] > t.max_count) t.max_count = t.count[g];
    }
    if (topo) *topo = t;
    return ROUTEPACK_OK;
}

// The device's default stream-ordered pool keeps the memory freed into it
// (release threshold: unlimited), set once per device: otherwise every
// synchronisation hands the pool's memory back and the next call maps it
// again, which costs milliseconds for the annealing state.
static void keep_pool_memory() {
    static std::atomic<uint64_t> done{0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return;
    if (done.fetch_or(1ull << dev) & (1ull << dev)) return;
    hipMemPool_t pool = nullptr;
    if (hipDeviceGetDefaultMemPool(&pool, dev) != hipSuccess || !pool) return;
    uint64_t threshold = UINT64_MAX;
    (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &threshold);
}

// One stream's scratch arena: [0, top) is held by the live Scratch objects
// on it (nested calls stack), want is the largest extent a call has needed.
struct Arena {
    char *base = nullptr;
    size_t cap = 0, top = 0, want = 0;
    int depth = 0;
    std::thread::id owner;
};

static std::mutex g_arena_mu;
static std::map<std::pair<int, hipStream_t>, Arena> g_arenas;  // (device, stream); never erased

Scratch::Scratch(hipStream_t s) : stream_(s) {
    keep_pool_memory();
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return;
    std::lock_guard<std::mutex> lock(g_arena_mu);
    Arena &a = g_arenas[std::make_pair(dev, s)];
    if (a.depth > 0 && a.owner != std::this_thread::get_id()) return;  // another thread's call: pool only
    a.owner = std::this_thread::get_id();
    depth_ = ++a.depth;
    start_ = a.top;
    arena_ = &a;
}

Scratch::~Scratch() {
    for (void *q : ptrs_) (void)hipFreeAsync(q, stream_);
    if (!arena_) return;
    std::lock_guard<std::mutex> lock(g_arena_mu);
    Arena &a = *arena_;
    constexpr size_t kGrain = (size_t)2 << 20;
    const size_t peak = (start_ + need_ + kGrain - 1) & ~(kGrain - 1);
    if (peak > a.want) a.want = peak;
    a.top = start_;
    --a.depth;
}

void *Scratch::alloc(size_t n) {
    n = (n + 255) & ~(size_t)255;
    if (arena_) {
        std::lock_guard<std::mutex> lock(g_arena_mu);
        Arena &a = *arena_;
        need_ += n;
        if (depth_ == a.depth) {  // the innermost live Scratch: the top of the arena is its own
            if (depth_ == 1 && a.top == 0 && a.want > a.cap) {
                // grow before the outermost call's first piece; the old arena
                // goes back to the pool in stream order
                if (a.base) (void)hipFreeAsync(a.base, stream_);
                a.base = nullptr;
                a.cap = 0;
                void *q = nullptr;
                if (hipMallocAsync(&q, a.want, stream_) == hipSuccess) {
                    a.base = static_cast<char *>(q);
                    a.cap = a.want;
                }
            }
            if (a.top + n <= a.cap) {
                void *q = a.base + a.top;
                a.top += n;
                return q;
            }
        }
    }
    void *q = nullptr;
    if (hipMallocAsync(&q, n, stream_) != hipSuccess) {
        failed_ = true;
        return nullptr;
    }
    ptrs_.push_back(q);
    return q;
}

// stats[0] sum t, [1] max t, [2] min t, [3] #{t > C/2}
__global__ void k_length_stats(const int32_t *__restrict__ t, int64_t n, int64_t cap,
                               unsigned long long *sum, long long *mx, long long *mn,
                               unsigned long long *big) {
    int64_t s = 0, b = 0;
    long long hi = LLONG_MIN, lo = LLONG_MAX;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t v = t[i];
        s += v;
        b += (2 * v > cap) ? 1 : 0;
        hi = v > hi ? v : hi;
        lo = v < lo ? v : lo;
    }
    s = wave_sum(s);
    b = wave_sum(b);
    hi = wave_max(hi);
    lo = wave_min(lo);
    if (lane_id() == 0) {
        atomicAdd(sum, (unsigned long long)s);
        atomicAdd(big, (unsigned long long)b);
        atomicMax(mx, hi);
        atomicMin(mn, lo);
    }
}

// tot[l] += sum_p q[i][l][p]; rate = max over rows of ceil(max_p q / t_i);
// neg set when any q < 0.
__global__ void k_layer_totals(const int32_t *__restrict__ q, const int32_t *__restrict__ t,
                               int64_t rows, int32_t L, int32_t P, unsigned long long *tot,
                               long long *rate, int32_t *neg) {
    long long rmax = 0;
    for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < rows;
         r += (int64_t)gridDim.x * blockDim.x) {
        const int32_t *row = q + r * P;
        int64_t s = 0, mx = 0;
        int bad = 0;
        for (int p = 0; p < P; ++p) {
            const int32_t v = row[p];
            s += v;
            mx = v > mx ? v : mx;
            bad |= (v < 0);
        }
        const int64_t ti = t[r / L];
        const long long rt = ti > 0 ? (mx + ti - 1) / ti : mx;
        rmax = rt > rmax ? rt : rmax;
        if (s) atomicAdd(&tot[r % L], (unsigned long long)s);
        if (bad) atomicOr(neg, 1);
    }
    rmax = wave_max(rmax);
    if (lane_id() == 0) atomicMax(rate, rmax);
}

__global__ void k_init_stats(unsigned long long *u, long long *mx, long long *mn, long long *rate,
                             int32_t *neg, int32_t L) {
    const int i = threadIdx.x;
    if (i < 2) u[i] = 0;
    if (i == 0) {
        *mx = LLONG_MIN;
        *mn = LLONG_MAX;
        *rate = 0;
        *neg = 0;
    }
    for (int l = i; l < L; l += blockDim.x) u[2 + l] = 0;
}

int window_stats(const routepack_problem *p, const int32_t *lengths, const int32_t *q,
                 WindowStats *out, hipStream_t stream) {
    const int32_t L = p->n_layers;
    Scratch scr(stream);
    // layout: u[0] sum, u[1] big, u[2..2+L) layer totals; then mx, mn, neg
    unsigned long long *u = scr.get<unsigned long long>(2 + L);
    long long *mm = scr.get<long long>(3);
    int32_t *neg = scr.get<int32_t>(1);
    if (scr.failed()) return ROUTEPACK_E_DEVICE;
    hipLaunchKernelGGL(k_init_stats, dim3(1), dim3(256), 0, stream, u, mm, mm + 1, mm + 2, neg, L);
    const int64_t n = p->n_samples;
    int blocks = (int)((n + 255) / 256);
    if (blocks > 1024) blocks = 1024;
    hipLaunchKernelGGL(k_length_stats, dim3(blocks), dim3(256), 0, stream, lengths, n,
                       (int64_t)p->capacity, u, mm, mm + 1, u + 1);
    if (q && L > 0) {
        const int64_t rows = n * L;
        int qb = (int)((rows + 255) / 256);
        if (qb > 4096) qb = 4096;
        hipLaunchKernelGGL(k_layer_totals, dim3(qb), dim3(256), 0, stream, q, lengths, rows, L,
                           p->n_ranks, u + 2, mm + 2, neg);
    }
    RP_HIP(hipGetLastError());
    std::vector<unsigned long long> hu(2 + L);
    long long hm[3];
    int32_t hneg = 0;
    RP_HIP(hipMemcpyAsync(hu.data(), u, sizeof(unsigned long long) * (2 + L),
                          hipMemcpyDeviceToHost, stream));
    RP_HIP(hipMemcpyAsync(hm, mm, sizeof(hm), hipMemcpyDeviceToHost, stream));
    RP_HIP(hipMemcpyAsync(&hneg, neg, sizeof(hneg), hipMemcpyDeviceToHost, stream));
    RP_HIP(hipStreamSynchronize(stream));
    out->sum_t = (int64_t)hu[0];
    out->n_big = (int64_t)hu[1];
    out->max_t = hm[0];
    out->min_t = hm[1];
    out->w_bound = 0;
    for (int l = 0; l < L; ++l)
        if ((int64_t)hu[2 + l] > out->w_bound) out->w_bound = (int64_t)hu[2 + l];
    out->q_negative = hneg != 0;
    out->q_rate = hm[2];
    return ROUTEPACK_OK;
}

int64_t w_entry_bound(const routepack_problem *p, const WindowStats &ws) {
    // A row-shard holds at most maxD * C tokens and q[i][l][p] <= rate * t_i.
    int32_t maxd = 0;
    {
        std::vector<int32_t> cnt(p->n_edp, 0);
        for (int d = 0; d < p->n_dp; ++d) cnt[p->dp_to_edp[d]]++;
        for (int g = 0; g < p->n_edp; ++g) maxd = cnt[g] > maxd ? cnt[g] : maxd;
    }
    const long double wcap = (long double)ws.q_rate * (long double)maxd * (long double)p->capacity;
    return wcap < (long double)ws.w_bound ? (int64_t)wcap : ws.w_bound;
}

int overflow_check(const routepack_problem *p, int64_t n_rows, const WindowStats &ws,
                   bool w_as_int32) {
    const long double lim = 9007199254740992.0L;  // 2^53
    const long double C = (long double)p->capacity;
    const int64_t wb = w_entry_bound(p, ws);
    long double a_max = 0.0L;
    for (int s = 0; s < p->n_stages; ++s)
        a_max += (long double)p->alpha_fp[s] * C + (long double)p->beta_fp[s] * C * C;
    const long double e_max = ldexpl((long double)p->n_layers * (long double)wb, p->frac_bits);
    const long double total = (long double)n_rows * (long double)p->n_edp * (a_max + e_max + 1.0L);
    if (!(total < lim)) return ROUTEPACK_E_OVERFLOW;
    if (!(ldexpl(C, p->frac_bits) < lim)) return ROUTEPACK_E_OVERFLOW;
    if (w_as_int32 && wb > 2147483647LL) return ROUTEPACK_E_OVERFLOW;
    return ROUTEPACK_OK;
}

int upload_problem(const routepack_problem *p, const Topology &topo, Scratch &scr,
                   DeviceProblem *dp, hipStream_t stream) {
    const int D = topo.D, G = topo.G, S = p->n_stages;
    dp->slots = scr.get<int32_t>((size_t)G * D);
    dp->count = scr.get<int32_t>(G);
    dp->slot_shard = scr.get<int32_t>(D);
    dp->alpha = scr.get<int64_t>(S);
    dp->beta = scr.get<int64_t>(S);
    if (scr.failed()) return ROUTEPACK_E_DEVICE;
    RP_HIP(hipMemcpyAsync(dp->slots, topo.slots.data(), sizeof(int32_t) * G * D,
                          hipMemcpyHostToDevice, stream));
    RP_HIP(hipMemcpyAsync(dp->count, topo.count.data(), sizeof(int32_t) * G,
                          hipMemcpyHostToDevice, stream));
    RP_HIP(hipMemcpyAsync(dp->slot_shard, p->dp_to_edp, sizeof(int32_t) * D,
                          hipMemcpyHostToDevice, stream));
    RP_HIP(hipMemcpyAsync(dp->alpha, p->alpha_fp, sizeof(int64_t) * S, hipMemcpyHostToDevice,
                          stream));
    RP_HIP(hipMemcpyAsync(dp->beta, p->beta_fp, sizeof(int64_t) * S, hipMemcpyHostToDevice,
                          stream));
    return ROUTEPACK_OK;
}

}  // namespace rp

extern "C" const char *routepack_strerror(int code) {
    switch (code) {
        case ROUTEPACK_OK: return "ok";
        case ROUTEPACK_E_INVALID: return "invalid argument";
        case ROUTEPACK_E_INFEASIBLE: return "infeasible window (t_i > C or too few samples for the row bound)";
        case ROUTEPACK_E_HEURISTIC: return "FixedRowFFD found no feasible row count";
        case ROUTEPACK_E_LAYOUT: return "layout violates coverage, capacity or non-empty cells";
        case ROUTEPACK_E_OVERFLOW: return "fixed-point score bound exceeds 2^53";
        case ROUTEPACK_E_DEVICE: return "HIP runtime error";
        case ROUTEPACK_E_INTERNAL: return "postcondition failed";
        case ROUTEPACK_E_UNSUPPORTED: return "size not supported by these kernels";
        default: return "unknown status";
    }
}
