// Exact objective of layouts (Eqs. cell-token-statistics, stage-aware-
// attention, row-expert-load, row-expert-cost, lexicographic-score) with
// feasibility status (Eqs. sample-bijection .. token-capacity) and the online
// load diagnostics (Eqs. global-ep-cv and ep-efficiency).
//
// Pass 1, one workgroup per (layout, row-shard h = r*G + g): scan the layout
// in 256-sample chunks, collect the chunk's members of h, add their q rows
// into the row-shard table W_h[L][P] (int64 in LDS; each thread owns fixed
// entries, so no atomics), and accumulate the cell statistics of h's cells.
// Then A(h), E(h) = 2^F sum_l max_p W_h, J(h), and per-layer max/sum of W_h
// for the diagnostics.  Pass 2, one workgroup per layout: the score tuple,
// status and diagnostics.
#include <math.h>

#include "rp_device.h"
#include "rp_internal.h"

namespace rp {

struct EvalArgs {
    const int32_t *t;        // [N]
    const int32_t *q;        // [N][L][P]
    const int32_t *layouts;  // [n][N]
    int32_t N, L, P, D, G, R, S, F;
    int64_t C;
    const int32_t *slots, *count, *slot_shard;
    const int64_t *alpha, *beta;
    int32_t *status;                        // [n]
    int64_t *Jbuf, *Abuf;                   // [n][R*G]
    int64_t *wmax, *wsum;                   // [n][R*G][L]
};

__global__ void __launch_bounds__(256) k_eval_rowshard(EvalArgs a) {
    extern __shared__ char smem[];
    const int64_t LP = (int64_t)a.L * a.P;
    const int64_t RG = (int64_t)a.R * a.G;
    int64_t *W = reinterpret_cast<int64_t *>(smem);     // [LP]
    int64_t *cT = W + LP;                               // [D] (only shard slots used)
    int64_t *cQ = cT + a.D;                             // [D]
    int32_t *cN = reinterpret_cast<int32_t *>(cQ + a.D);  // [D]
    int32_t *mem = cN + a.D;                            // [256]
    int32_t *nmem = mem + 256;                          // [1]
    int32_t *stat = nmem + 1;                           // [1]
    int64_t *red = reinterpret_cast<int64_t *>(((uintptr_t)(stat + 1) + 7) & ~(uintptr_t)7);  // [4]

    const int64_t lay_idx = blockIdx.x / RG;
    const int64_t h = blockIdx.x % RG;
    const int32_t r = (int32_t)(h / a.G), g = (int32_t)(h % a.G);
    const int32_t *lay = a.layouts + lay_idx * a.N;
    const int64_t B = (int64_t)a.R * a.D;
    const int tid = threadIdx.x;

    for (int64_t e = tid; e < LP; e += blockDim.x) W[e] = 0;
    for (int d = tid; d < a.D; d += blockDim.x) {
        cT[d] = 0;
        cQ[d] = 0;
        cN[d] = 0;
    }
    if (tid == 0) {
        *nmem = 0;
        *stat = 0;
    }
    __syncthreads();
    for (int64_t base = 0; base < a.N; base += blockDim.x) {
        const int64_t i = base + tid;
        if (i < a.N) {
            const int32_t c = lay[i];
            if (c < 0 || c >= B) {
                if (h == 0) atomicOr(stat, 1);
            } else if (c / a.D == r && a.slot_shard[c % a.D] == g) {
                const int d = c % a.D;
                const int64_t ti = a.t[i];
                atomicAdd(reinterpret_cast<unsigned long long *>(&cT[d]), (unsigned long long)ti);
                atomicAdd(reinterpret_cast<unsigned long long *>(&cQ[d]), (unsigned long long)(ti * ti));
                atomicAdd(&cN[d], 1);
                mem[atomicAdd(nmem, 1)] = (int32_t)i;
            }
        }
        __syncthreads();
        const int32_t nm = *nmem;
        for (int32_t m = 0; m < nm; ++m) {
            const int32_t *qi = a.q + (int64_t)mem[m] * LP;
            for (int64_t e = tid; e < LP; e += blockDim.x) W[e] += qi[e];
        }
        __syncthreads();
        if (tid == 0) *nmem = 0;
        __syncthreads();
    }
    // Per-layer max and sum of W_h; E = 2^F sum_l max_p W.
    int64_t esum = 0;
    for (int l = tid; l < a.L; l += blockDim.x) {
        int64_t mx = W[(int64_t)l * a.P], sm = 0;
        for (int p = 0; p < a.P; ++p) {
            const int64_t v = W[(int64_t)l * a.P + p];
            mx = v > mx ? v : mx;
            sm += v;
        }
        esum += mx;
        const int64_t o = (lay_idx * RG + h) * a.L + l;
        a.wmax[o] = mx;
        a.wsum[o] = sm;
    }
    esum = wave_sum(esum);
    if (lane_id() == 0) red[wave_id()] = esum;
    __syncthreads();
    if (tid == 0) {
        int64_t e = 0;
        for (int w = 0; w < (int)(blockDim.x / kWave); ++w) e += red[w];
        int32_t st = *stat;
        int64_t A = 0;
        const int32_t m = a.count[g];
        for (int s = 0; s < a.S; ++s) {
            int64_t mx = 0;
            for (int x = 0; x < m; ++x) {
                const int d = a.slots[g * a.D + x];
                const int64_t cost = a.alpha[s] * cT[d] + a.beta[s] * cQ[d];
                if (x == 0 || cost > mx) mx = cost;
            }
            A += mx;
        }
        for (int x = 0; x < m; ++x) {
            const int d = a.slots[g * a.D + x];
            if (cT[d] > a.C) st |= 2;
            if (cN[d] == 0) st |= 4;
        }
        if (st) atomicOr(&a.status[lay_idx], st);
        a.Abuf[lay_idx * RG + h] = A;
        a.Jbuf[lay_idx * RG + h] = A + (e << a.F);
    }
}

__device__ inline double wave_sum_d(double v) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, kWave);
    return v;
}
__device__ inline double wave_max_d(double v) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        const double o = __shfl_xor(v, d, kWave);
        v = o > v ? o : v;
    }
    return v;
}

struct FinalArgs {
    int32_t L, P, G, R;
    double scale;
    const int32_t *status;
    const int64_t *Jbuf, *Abuf, *wmax, *wsum;
    const int64_t *rank_load;  // [L][P] or null
    int64_t *scores;           // [n][3]
    int64_t *J;                // [n][RG] or null
    double *diag;              // [n][8] or null
};

__global__ void __launch_bounds__(256) k_eval_finalize(FinalArgs a) {
    __shared__ int64_t ri[3][4];
    __shared__ double rd[4][4];
    const int64_t lay = blockIdx.x;
    const int64_t RG = (int64_t)a.R * a.G;
    const int tid = threadIdx.x, lane = lane_id(), wv = wave_id();
    const int64_t *Jl = a.Jbuf + lay * RG;
    const int32_t st = a.status[lay];
    // U_g = sum_r J(r, g): s0 = max_g U, s1 = sum_g U; s2 = max J.
    int64_t umax = LLONG_MIN, usum = 0, jmax = LLONG_MIN;
    for (int g = tid; g < a.G; g += blockDim.x) {
        int64_t U = 0;
        for (int r = 0; r < a.R; ++r) U += Jl[(int64_t)r * a.G + g];
        umax = U > umax ? U : umax;
        usum += U;
    }
    for (int64_t h = tid; h < RG; h += blockDim.x) jmax = Jl[h] > jmax ? Jl[h] : jmax;
    umax = wave_max(umax);
    usum = wave_sum(usum);
    jmax = wave_max(jmax);
    if (lane == 0) {
        ri[0][wv] = umax;
        ri[1][wv] = usum;
        ri[2][wv] = jmax;
    }
    // Diagnostics partials.
    double cv = 0.0, sep = 0.0, tep = 0.0, ideal = 0.0, att = 0.0;
    if (a.diag) {
        if (a.rank_load) {
            for (int l = tid; l < a.L; l += blockDim.x) {
                double mean = 0.0;
                for (int p = 0; p < a.P; ++p) mean += (double)a.rank_load[(int64_t)l * a.P + p];
                mean /= (double)a.P;
                double var = 0.0;
                for (int p = 0; p < a.P; ++p) {
                    const double dv = (double)a.rank_load[(int64_t)l * a.P + p] - mean;
                    var += dv * dv;
                }
                var /= (double)a.P;
                cv += mean > 0.0 ? sqrt(var) / mean : 0.0;
            }
        }
        for (int64_t x = tid; x < (int64_t)a.R * a.L; x += blockDim.x) {
            const int64_t r = x / a.L, l = x % a.L;
            int64_t mx = 0;
            double best_mean = 0.0;
            for (int g = 0; g < a.G; ++g) {
                const int64_t o = ((lay * RG) + r * a.G + g) * a.L + l;
                mx = a.wmax[o] > mx ? a.wmax[o] : mx;
                const double mean = (double)a.wsum[o] / (double)a.P;
                best_mean = mean > best_mean ? mean : best_mean;
            }
            sep += (double)mx;
            tep = (double)mx > tep ? (double)mx : tep;
            ideal += best_mean;
        }
        for (int64_t h = tid; h < RG; h += blockDim.x) att += (double)a.Abuf[lay * RG + h] / a.scale;
        cv = wave_sum_d(cv);
        sep = wave_sum_d(sep);
        tep = wave_max_d(tep);
        ideal = wave_sum_d(ideal);
        att = wave_sum_d(att);
        if (lane == 0) {
            rd[0][wv] = cv;
            rd[1][wv] = sep;
            rd[2][wv] = tep;
            rd[3][wv] = ideal;
        }
        __shared__ double ra[4];
        if (lane == 0) ra[wv] = att;
        __syncthreads();
        if (tid == 0) {
            double s_cv = 0, s_sep = 0, s_tep = 0, s_ideal = 0, s_att = 0;
            for (int w = 0; w < (int)(blockDim.x / kWave); ++w) {
                s_cv += rd[0][w];
                s_sep += rd[1][w];
                s_tep = rd[2][w] > s_tep ? rd[2][w] : s_tep;
                s_ideal += rd[3][w];
                s_att += ra[w];
            }
            int64_t s0 = LLONG_MIN, s1 = 0, s2 = LLONG_MIN;
            for (int w = 0; w < (int)(blockDim.x / kWave); ++w) {
                s0 = ri[0][w] > s0 ? ri[0][w] : s0;
                s1 += ri[1][w];
                s2 = ri[2][w] > s2 ? ri[2][w] : s2;
            }
            double *dg = a.diag + lay * 8;
            if (st) {
                for (int k = 0; k < 8; ++k) dg[k] = __builtin_nan("");
            } else {
                dg[0] = a.rank_load ? (a.L > 0 ? s_cv / (double)a.L : 0.0) : __builtin_nan("");
                dg[1] = s_sep;
                dg[2] = s_tep;
                dg[3] = s_sep > 0.0 ? s_ideal / s_sep : 1.0;
                dg[4] = s_att;
                dg[5] = (double)s0 / a.scale;
                dg[6] = (double)s1 / a.scale;
                dg[7] = energy(s0, s1, s2, a.scale);
            }
        }
    }
    __syncthreads();
    if (tid == 0) {
        int64_t s0 = LLONG_MIN, s1 = 0, s2 = LLONG_MIN;
        for (int w = 0; w < (int)(blockDim.x / kWave); ++w) {
            s0 = ri[0][w] > s0 ? ri[0][w] : s0;
            s1 += ri[1][w];
            s2 = ri[2][w] > s2 ? ri[2][w] : s2;
        }
        int64_t *so = a.scores + lay * 3;
        if (st) {
            so[0] = so[1] = so[2] = LLONG_MAX;
        } else {
            so[0] = s0;
            so[1] = s1;
            so[2] = s2;
        }
    }
    if (a.J)
        for (int64_t h = tid; h < RG; h += blockDim.x) a.J[lay * RG + h] = st ? LLONG_MAX : Jl[h];
}

__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t v) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

// Scores `n` layouts already on the device; used by the public entry point
// and by the packing path.  status must hold n int32.
int eval_layouts(const routepack_problem *p, const Topology &topo, const DeviceProblem &dp,
                 const int32_t *t, const int32_t *q, int32_t R, int64_t n, const int32_t *layouts,
                 int64_t *scores, int32_t *status, int64_t *J, double *diag,
                 const int64_t *rank_load, hipStream_t stream) {
    if (n == 0) return ROUTEPACK_OK;
    const int64_t RG = (int64_t)R * topo.G, LP = (int64_t)p->n_layers * p->n_ranks;
    if (LP > 16384) return ROUTEPACK_E_UNSUPPORTED;
    Scratch scr(stream);
    int64_t *Jbuf = scr.get<int64_t>(n * RG);
    int64_t *Abuf = scr.get<int64_t>(n * RG);
    int64_t *wmax = scr.get<int64_t>(n * RG * (p->n_layers ? p->n_layers : 1));
    int64_t *wsum = scr.get<int64_t>(n * RG * (p->n_layers ? p->n_layers : 1));
    if (scr.failed()) return ROUTEPACK_E_DEVICE;
    hipLaunchKernelGGL(k_fill_i32, dim3((unsigned)((n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024)),
                       dim3(256), 0, stream, status, n, 0);
    EvalArgs a;
    a.t = t; a.q = q; a.layouts = layouts;
    a.N = p->n_samples; a.L = p->n_layers; a.P = p->n_ranks; a.D = topo.D; a.G = topo.G; a.R = R;
    a.S = p->n_stages; a.F = p->frac_bits; a.C = p->capacity;
    a.slots = dp.slots; a.count = dp.count; a.slot_shard = dp.slot_shard;
    a.alpha = dp.alpha; a.beta = dp.beta;
    a.status = status; a.Jbuf = Jbuf; a.Abuf = Abuf; a.wmax = wmax; a.wsum = wsum;
    const size_t lds = (size_t)LP * 8 + (size_t)topo.D * 20 + 256 * 4 + 64 + 64;
    if (lds > 160 * 1024) return ROUTEPACK_E_UNSUPPORTED;
    hipLaunchKernelGGL(k_eval_rowshard, dim3((unsigned)(n * RG)), dim3(256), lds, stream, a);
    FinalArgs f;
    f.L = p->n_layers; f.P = p->n_ranks; f.G = topo.G; f.R = R;
    f.scale = ldexp((double)p->capacity, p->frac_bits);
    f.status = status; f.Jbuf = Jbuf; f.Abuf = Abuf; f.wmax = wmax; f.wsum = wsum;
    f.rank_load = rank_load; f.scores = scores; f.J = J; f.diag = diag;
    hipLaunchKernelGGL(k_eval_finalize, dim3((unsigned)n), dim3(256), 0, stream, f);
    RP_HIP(hipGetLastError());
    return ROUTEPACK_OK;
}

}  // namespace rp

using namespace rp;

extern "C" int routepack_eval_objective(const routepack_problem *prob, const int32_t *lengths,
                                        const int32_t *q, int32_t n_rows, int32_t n_layouts,
                                        const int32_t *layouts, int64_t *scores, int32_t *status,
                                        int64_t *J, double *diag, const int64_t *rank_load,
                                        hipStream_t stream) {
    Topology topo;
    RP_TRY(check_problem(prob, &topo));
    if (n_rows < 1 || n_layouts < 0) return ROUTEPACK_E_INVALID;
    if (!lengths || (!q && prob->n_layers > 0) || !scores || !status || (!layouts && n_layouts > 0))
        return ROUTEPACK_E_INVALID;
    WindowStats ws;
    RP_TRY(window_stats(prob, lengths, q, &ws, stream));
    if (ws.min_t < 1 || ws.q_negative) return ROUTEPACK_E_INVALID;
    RP_TRY(overflow_check(prob, n_rows, ws, false));
    Scratch scr(stream);
    DeviceProblem dp;
    RP_TRY(upload_problem(prob, topo, scr, &dp, stream));
    RP_TRY(eval_layouts(prob, topo, dp, lengths, q, n_rows, n_layouts, layouts, scores, status, J,
                        diag, rank_load, stream));
    RP_HIP(hipStreamSynchronize(stream));
    return ROUTEPACK_OK;
}
