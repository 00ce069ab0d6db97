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
    if ((m >> 32) == 0) {
        // m < 2^32: w m = hi(w) m 2^32 + lo(w) m, and adding
        // floor(lo(w) m / 2^32) before the shift gives the same floor; both
        // products are 32 x 32 -> 64 and the sum stays below 2^64.
        const uint64_t a = (w >> 32) * m, b = (w & 0xFFFFFFFFull) * m;
        return (a + (b >> 32)) >> 32;
    }
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
// wave64 collectives (every lane of the wave participates).  Reductions and
// scans use DPP row operations (16-lane rows) and combine the four rows with
// readlane, so the full-wave results are uniform scalars; no LDS traffic.
__device__ inline int lane_id() { return (int)(threadIdx.x & (kWave - 1)); }
__device__ inline int wave_id() { return (int)(threadIdx.x / kWave); }

// DPP controls (GFX9 encoding).
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;  // reverse within 8 lanes
constexpr int kDppMirror = 0x140;      // reverse within 16 lanes
constexpr int kDppRowShr1 = 0x111;
constexpr int kDppRowBcast15 = 0x142;
constexpr int kDppRowBcast31 = 0x143;

template <int CTRL, int ROW_MASK = 0xF>
__device__ inline int32_t dpp32(int32_t v, int32_t old) {
    return __builtin_amdgcn_update_dpp(old, v, CTRL, ROW_MASK, 0xF, false);
}
template <int CTRL, int ROW_MASK = 0xF>
__device__ inline int64_t dpp64(int64_t v, int64_t old) {
    const int32_t lo = dpp32<CTRL, ROW_MASK>((int32_t)(uint32_t)v, (int32_t)(uint32_t)old);
    const int32_t hi = dpp32<CTRL, ROW_MASK>((int32_t)(uint32_t)((uint64_t)v >> 32),
                                             (int32_t)(uint32_t)((uint64_t)old >> 32));
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

__device__ inline uint64_t readlane64(uint64_t v, int lane) {
    const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)v, lane);
    const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane);
    return ((uint64_t)hi << 32) | lo;
}

// Row (16-lane) reductions: every lane ends with its row's result.
__device__ inline int64_t row_max64(int64_t v) {
    int64_t o;
    o = dpp64<kDppXor1>(v, v); v = o > v ? o : v;
    o = dpp64<kDppXor2>(v, v); v = o > v ? o : v;
    o = dpp64<kDppHalfMirror>(v, v); v = o > v ? o : v;
    o = dpp64<kDppMirror>(v, v); v = o > v ? o : v;
    return v;
}
__device__ inline int64_t row_min64(int64_t v) {
    int64_t o;
    o = dpp64<kDppXor1>(v, v); v = o < v ? o : v;
    o = dpp64<kDppXor2>(v, v); v = o < v ? o : v;
    o = dpp64<kDppHalfMirror>(v, v); v = o < v ? o : v;
    o = dpp64<kDppMirror>(v, v); v = o < v ? o : v;
    return v;
}
__device__ inline int32_t row_sum32(int32_t v) {
    v += dpp32<kDppXor1>(v, 0);
    v += dpp32<kDppXor2>(v, 0);
    v += dpp32<kDppHalfMirror>(v, 0);
    v += dpp32<kDppMirror>(v, 0);
    return v;
}
__device__ inline int64_t row_sum64(int64_t v) {
    v += dpp64<kDppXor1>(v, 0);
    v += dpp64<kDppXor2>(v, 0);
    v += dpp64<kDppHalfMirror>(v, 0);
    v += dpp64<kDppMirror>(v, 0);
    return v;
}

__device__ inline int64_t wave_sum(int64_t v) {
    v = row_sum64(v);
    return (int64_t)(readlane64((uint64_t)v, 0) + readlane64((uint64_t)v, 16) +
                     readlane64((uint64_t)v, 32) + readlane64((uint64_t)v, 48));
}
__device__ inline int64_t wave_max(int64_t v) {
    v = row_max64(v);
    int64_t a = (int64_t)readlane64((uint64_t)v, 0), b = (int64_t)readlane64((uint64_t)v, 16);
    int64_t c = (int64_t)readlane64((uint64_t)v, 32), d = (int64_t)readlane64((uint64_t)v, 48);
    a = b > a ? b : a;
    c = d > c ? d : c;
    return c > a ? c : a;
}
__device__ inline int64_t wave_min(int64_t v) {
    v = row_min64(v);
    int64_t a = (int64_t)readlane64((uint64_t)v, 0), b = (int64_t)readlane64((uint64_t)v, 16);
    int64_t c = (int64_t)readlane64((uint64_t)v, 32), d = (int64_t)readlane64((uint64_t)v, 48);
    a = b < a ? b : a;
    c = d < c ? d : c;
    return c < a ? c : a;
}
__device__ inline int32_t wave_max32(int32_t v) {
    int32_t o;
    o = dpp32<kDppXor1>(v, v); v = o > v ? o : v;
    o = dpp32<kDppXor2>(v, v); v = o > v ? o : v;
    o = dpp32<kDppHalfMirror>(v, v); v = o > v ? o : v;
    o = dpp32<kDppMirror>(v, v); v = o > v ? o : v;
    int32_t a = __builtin_amdgcn_readlane(v, 0), b = __builtin_amdgcn_readlane(v, 16);
    int32_t c = __builtin_amdgcn_readlane(v, 32), d = __builtin_amdgcn_readlane(v, 48);
    a = b > a ? b : a;
    c = d > c ? d : c;
    return c > a ? c : a;
}

// Inclusive prefix sum over the 64 lanes: row scans by row_shr 1, 2, 4, 8,
// then the row totals carried across rows by row_bcast15 and row_bcast31.
__device__ inline int64_t wave_incl_scan(int64_t v) {
    v += dpp64<kDppRowShr1>(v, 0);
    v += dpp64<kDppRowShr1 + 1>(v, 0);
    v += dpp64<kDppRowShr1 + 3>(v, 0);
    v += dpp64<kDppRowShr1 + 7>(v, 0);
    v += dpp64<kDppRowBcast15, 0xA>(v, 0);
    v += dpp64<kDppRowBcast31, 0xC>(v, 0);
    return v;
}
__device__ inline uint64_t wave_incl_scan_u(uint64_t v) {
    return (uint64_t)wave_incl_scan((int64_t)v);
}

// Maximum over aligned groups of P adjacent lanes (P a power of two <= 64);
// every lane of a group ends with the group's maximum.
__device__ inline int32_t seg_max32(int32_t v, int P) {
    int32_t o;
    if (P >= 2) { o = dpp32<kDppXor1>(v, v); v = o > v ? o : v; }
    if (P >= 4) { o = dpp32<kDppXor2>(v, v); v = o > v ? o : v; }
    if (P >= 8) { o = dpp32<kDppHalfMirror>(v, v); v = o > v ? o : v; }
    if (P >= 16) { o = dpp32<kDppMirror>(v, v); v = o > v ? o : v; }
    if (P >= 32) {  // swap 16-lane halves of each 32-lane group
        o = __builtin_amdgcn_ds_swizzle(v, 0x401F);
        v = o > v ? o : v;
    }
    if (P >= 64) {
        o = __shfl_xor(v, 32, kWave);
        v = o > v ? o : v;
    }
    return v;
}

template <int CTRL>
__device__ inline void lexmin_step(int64_t &k0, int64_t &k1, int64_t &k2, int64_t &kj) {
    const int64_t o0 = dpp64<CTRL>(k0, k0), o1 = dpp64<CTRL>(k1, k1);
    const int64_t o2 = dpp64<CTRL>(k2, k2), oj = dpp64<CTRL>(kj, kj);
    if (lex_less(o0, o1, o2, k0, k1, k2) || (o0 == k0 && o1 == k1 && o2 == k2 && oj < kj)) {
        k0 = o0;
        k1 = o1;
        k2 = o2;
        kj = oj;
    }
}

// Lexicographic minimum of (k0, k1, k2) over the wave, lowest kj on ties;
// the result is uniform.
__device__ inline void wave_lexmin(int64_t &k0, int64_t &k1, int64_t &k2, int64_t &kj) {
    lexmin_step<kDppXor1>(k0, k1, k2, kj);
    lexmin_step<kDppXor2>(k0, k1, k2, kj);
    lexmin_step<kDppHalfMirror>(k0, k1, k2, kj);
    lexmin_step<kDppMirror>(k0, k1, k2, kj);
    int64_t b0 = (int64_t)readlane64((uint64_t)k0, 0), b1 = (int64_t)readlane64((uint64_t)k1, 0);
    int64_t b2 = (int64_t)readlane64((uint64_t)k2, 0), bj = (int64_t)readlane64((uint64_t)kj, 0);
#pragma unroll
    for (int row = 1; row < 4; ++row) {
        const int64_t o0 = (int64_t)readlane64((uint64_t)k0, 16 * row), o1 = (int64_t)readlane64((uint64_t)k1, 16 * row);
        const int64_t o2 = (int64_t)readlane64((uint64_t)k2, 16 * row), oj = (int64_t)readlane64((uint64_t)kj, 16 * row);
        if (lex_less(o0, o1, o2, b0, b1, b2) || (o0 == b0 && o1 == b1 && o2 == b2 && oj < bj)) {
            b0 = o0;
            b1 = o1;
            b2 = o2;
            bj = oj;
        }
    }
    k0 = b0;
    k1 = b1;
    k2 = b2;
    kj = bj;
}

// Unsigned 64-bit maximum over the wave; uniform.
__device__ inline uint64_t wave_max_u64(uint64_t v) {
    uint64_t o;
    o = (uint64_t)dpp64<kDppXor1>((int64_t)v, (int64_t)v); v = o > v ? o : v;
    o = (uint64_t)dpp64<kDppXor2>((int64_t)v, (int64_t)v); v = o > v ? o : v;
    o = (uint64_t)dpp64<kDppHalfMirror>((int64_t)v, (int64_t)v); v = o > v ? o : v;
    o = (uint64_t)dpp64<kDppMirror>((int64_t)v, (int64_t)v); v = o > v ? o : v;
    uint64_t a = readlane64(v, 0), b = readlane64(v, 16), c = readlane64(v, 32), d = readlane64(v, 48);
    a = b > a ? b : a;
    c = d > c ? d : c;
    return c > a ? c : a;
}

__device__ inline int first_lane(uint64_t mask) { return mask ? __ffsll((long long)mask) - 1 : -1; }

}  // namespace rp
