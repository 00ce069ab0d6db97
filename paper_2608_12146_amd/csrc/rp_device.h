// Device-side building blocks shared by the gfx950 kernels of the RoutePack
// hot path: counter-based Philox4x64-10, bounded draws, a deterministic exp,
// the annealing energy, lexicographic score comparison, and wave64
// reductions/scans.  Everything that decides an accept or a resampling
// parent is integer arithmetic or a fixed sequence of IEEE binary64
// operations; the translation units are compiled with -ffp-contract=off so
// no multiply-add is fused.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#pragma clang fp contract(off)

namespace rp {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11).  Round: the 128-bit
// products of counter words 0 and 2 with the two multipliers; new counter =
// (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0); the key advances by the Weyl
// increments between rounds.
struct U64x4 {
    uint64_t v[4];
};

__host__ __device__ inline U64x4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2,
                                               uint64_t c3, uint64_t k0, uint64_t k1) {
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
#if defined(__HIP_DEVICE_COMPILE__)
        const uint64_t hi0 = __umul64hi(M0, c0), lo0 = M0 * c0;
        const uint64_t hi1 = __umul64hi(M1, c2), lo1 = M1 * c2;
#else
        const unsigned __int128 p0 = (unsigned __int128)M0 * c0, p1 = (unsigned __int128)M1 * c2;
        const uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
        const uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
#endif
        const uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
        k0 += W0;
        k1 += W1;
    }
    U64x4 o;
    o.v[0] = c0; o.v[1] = c1; o.v[2] = c2; o.v[3] = c3;
    return o;
}

// floor(w * m / 2^64): the multiply-shift bounded draw.
__host__ __device__ inline uint64_t bounded(uint64_t w, uint64_t m) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __umul64hi(w, m);
#else
    return (uint64_t)(((unsigned __int128)w * m) >> 64);
#endif
}

// ---------------------------------------------------------------------------
// exp(x) for x <= 0 with a result that depends only on IEEE binary64
// rounding: Cody-Waite reduction x = k*ln2 + r (ln2 split into a head with 32
// significant bits and a tail), Horner evaluation of sum_{m<=13} r^m / m!
// with each coefficient the double nearest 1/m!, then scaling by 2^k (exact:
// for x >= -708 the result is a normal double).
__host__ __device__ inline double exp_det(double x) {
    const double kInvLn2 = 1.44269504088896338700e+00;
    const double kLn2Hi = 6.93147180369123816490e-01;
    const double kLn2Lo = 1.90821492927058770002e-10;
    if (!(x >= -708.0)) return 0.0;
    if (x > 0.0) x = 0.0;
    const double k = __builtin_rint(x * kInvLn2);
    const double r = (x - k * kLn2Hi) - k * kLn2Lo;
    double p = 1.0 / 6227020800.0;
    p = p * r + 1.0 / 479001600.0;
    p = p * r + 1.0 / 39916800.0;
    p = p * r + 1.0 / 3628800.0;
    p = p * r + 1.0 / 362880.0;
    p = p * r + 1.0 / 40320.0;
    p = p * r + 1.0 / 5040.0;
    p = p * r + 1.0 / 720.0;
    p = p * r + 1.0 / 120.0;
    p = p * r + 1.0 / 24.0;
    p = p * r + 1.0 / 6.0;
    p = p * r + 0.5;
    p = p * r + 1.0;
    p = p * r + 1.0;
    return __builtin_ldexp(p, (int)k);
}

// Annealing energy (Eq. pa-energy) of a fixed-point score, with
// S_i = s_i / (2^F C) correctly rounded.
__host__ __device__ inline double energy(int64_t s0, int64_t s1, int64_t s2, double scale) {
    const double e0 = (double)s0 / scale, e1 = (double)s1 / scale, e2 = (double)s2 / scale;
    const double a = e0 + 1e-6 * e1;
    return a + 1e-9 * e2;
}

__host__ __device__ inline bool lex_less(int64_t a0, int64_t a1, int64_t a2, int64_t b0,
                                         int64_t b1, int64_t b2) {
    if (a0 != b0) return a0 < b0;
    if (a1 != b1) return a1 < b1;
    return a2 < b2;
}

// ---------------------------------------------------------------------------
// wave64 collectives (every lane of the wave participates).
__device__ inline int lane_id() { return (int)(threadIdx.x & (kWave - 1)); }
__device__ inline int wave_id() { return (int)(threadIdx.x / kWave); }

__device__ inline int64_t wave_sum(int64_t v) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, kWave);
    return v;
}
__device__ inline int64_t wave_max(int64_t v) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        const int64_t o = __shfl_xor(v, d, kWave);
        v = o > v ? o : v;
    }
    return v;
}
__device__ inline int64_t wave_min(int64_t v) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        const int64_t o = __shfl_xor(v, d, kWave);
        v = o < v ? o : v;
    }
    return v;
}
__device__ inline int32_t wave_max32(int32_t v) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        const int32_t o = __shfl_xor(v, d, kWave);
        v = o > v ? o : v;
    }
    return v;
}
// inclusive prefix sum over lanes
__device__ inline int64_t wave_incl_scan(int64_t v) {
    const int lane = lane_id();
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const int64_t o = __shfl_up(v, d, kWave);
        if (lane >= d) v += o;
    }
    return v;
}
__device__ inline uint64_t wave_incl_scan_u(uint64_t v) {
    const int lane = lane_id();
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const uint64_t o = __shfl_up(v, d, kWave);
        if (lane >= d) v += o;
    }
    return v;
}
__device__ inline int first_lane(uint64_t mask) { return mask ? __ffsll((long long)mask) - 1 : -1; }

}  // namespace rp
