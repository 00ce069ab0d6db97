// Host-side internals of the RoutePack C-ABI library: argument validation,
// topology tables, HIP error mapping, stream-ordered scratch, and the window
// bounds that guard the fixed-point arithmetic.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "routepack.h"

namespace rp {

#define RP_HIP(call)                                         \
    do {                                                     \
        hipError_t _e = (call);                              \
        if (_e != hipSuccess) return ROUTEPACK_E_DEVICE;     \
    } while (0)

#define RP_TRY(call)                  \
    do {                              \
        int _rc = (call);             \
        if (_rc != ROUTEPACK_OK) return _rc; \
    } while (0)

// Slots of each EDP shard in ascending order, packed for kernels:
// slots[g * D + x] is the x-th slot of shard g, count[g] its size.
struct Topology {
    int32_t D = 0, G = 0;
    std::vector<int32_t> count, slots;
    int32_t max_count = 0;
};

// Validates the sizes, coefficients and partition of a problem.
int check_problem(const routepack_problem *p, Topology *topo);

struct Arena;

// RAII device scratch for one call on one stream.  Each (device, stream)
// keeps an arena that the innermost live Scratch on it bump-allocates from;
// the arena is sized to the largest total a call on that stream has asked
// for and is reused by the next call (the stream orders the calls), so a
// call costs no allocator round trips once the stream has seen its size.
// What does not fit comes from the device's stream-ordered pool and goes
// back to it when the Scratch ends.  Nothing is allocated before the first
// alloc().  An arena lives until the process ends.
class Scratch {
  public:
    explicit Scratch(hipStream_t s);
    ~Scratch();
    Scratch(const Scratch &) = delete;
    Scratch &operator=(const Scratch &) = delete;
    // Allocates n bytes (256-byte aligned); returns nullptr on failure.
    void *alloc(size_t n);
    template <class T>
    T *get(size_t count) { return static_cast<T *>(alloc(sizeof(T) * (count ? count : 1))); }
    bool failed() const { return failed_; }

  private:
    hipStream_t stream_;
    Arena *arena_ = nullptr;  // this stream's arena (null: another thread holds it)
    int depth_ = 0;           // nesting depth of this Scratch on the arena
    size_t start_ = 0;        // arena offset when this Scratch began
    size_t need_ = 0;         // bytes this Scratch asked for
    std::vector<void *> ptrs_;  // pieces taken from the pool
    bool failed_ = false;
};

// Bounds of one window, computed on the device and read back.
struct WindowStats {
    int64_t sum_t = 0, max_t = 0, min_t = 0, n_big = 0;  // n_big: t_i > C/2
    int64_t w_bound = 0;                                  // max_l sum_{i,p} q[i][l][p]
    int64_t q_rate = 0;                                   // max_i ceil(max_{l,p} q[i][l][p] / t_i)
    bool q_negative = false;
};
int window_stats(const routepack_problem *p, const int32_t *lengths, const int32_t *q,
                 WindowStats *out, hipStream_t stream);
// Bound of every W entry of a capacity-feasible layout: min(w_bound, q_rate * maxD * C).
int64_t w_entry_bound(const routepack_problem *p, const WindowStats &ws);

// R * G * (A_max + E_max + 1) < 2^53 and 2^F * C < 2^53 (scores exact in
// int64 and as doubles), with W bounded by min(w_bound, q_rate * maxD * C)
// for capacity-feasible layouts; W entries must also fit int32 when
// w_as_int32.
int overflow_check(const routepack_problem *p, int64_t n_rows, const WindowStats &ws,
                   bool w_as_int32);

// sigma = the samples ordered by (-t, i) (rp_pack.hip).
int rank_sort_desc(const int32_t *lengths, int32_t N, int32_t *sigma, hipStream_t stream);

// Device copies of small per-problem tables.
struct DeviceProblem {
    int32_t *slots = nullptr;   // [G][D]
    int32_t *count = nullptr;   // [G]
    int32_t *slot_shard = nullptr;  // [D] = dp_to_edp
    int64_t *alpha = nullptr, *beta = nullptr;  // [S]
};
int upload_problem(const routepack_problem *p, const Topology &topo, Scratch &scr,
                   DeviceProblem *dp, hipStream_t stream);

}  // namespace rp
