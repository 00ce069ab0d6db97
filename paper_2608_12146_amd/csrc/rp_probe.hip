// LDS read-bandwidth probe (a measurement aid; see routepack_probe.h).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "routepack.h"
#include "routepack_probe.h"

namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeWords = 4096;  // 16-byte words: 64 KiB of LDS per workgroup

__global__ void __launch_bounds__(kProbeThreads) k_lds_read(int32_t reps, uint32_t *sink) {
    __shared__ ulonglong2 buf[kProbeWords];
    const int t = threadIdx.x;
    for (int x = t; x < kProbeWords; x += kProbeThreads)
        buf[x] = make_ulonglong2((uint64_t)x * 0x9E3779B97F4A7C15ull, (uint64_t)x * 0xC2B2AE3D27D4EB4Full);
    __syncthreads();
    // Step r reads word (t + 256 r) mod 4096: the 16 steps of a period sit at
    // fixed offsets from the thread's first word, so a period is 16 reads
    // with immediate offsets and two 64-bit adds each; the base is made
    // opaque per period so the reads are not hoisted out of the loop.
    uint64_t a0 = 0, a1 = 0;
    int32_t off = t * 16;
    int32_t r = 0;
    for (; r + 16 <= reps; r += 16) {
        asm volatile("" : "+v"(off));
        const char *p = reinterpret_cast<const char *>(buf) + off;
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            const ulonglong2 v = *reinterpret_cast<const ulonglong2 *>(p + u * 4096);
            a0 += v.x;
            a1 += v.y;
        }
    }
    for (; r < reps; ++r) {
        const ulonglong2 v = buf[(t + kProbeThreads * (r & 15)) & (kProbeWords - 1)];
        a0 += v.x;
        a1 += v.y;
    }
    const uint64_t sum = a0 + a1;
    sink[(int64_t)blockIdx.x * kProbeThreads + t] = (uint32_t)(sum ^ (sum >> 32));
}

}  // namespace

extern "C" int routepack_probe_lds_read(int32_t n_workgroups, int32_t reps, uint32_t *sink, double *ms,
                                        int64_t *bytes, hipStream_t stream) {
    if (!sink || !ms || !bytes || n_workgroups < 1 || reps < 1) return ROUTEPACK_E_INVALID;
    if ((int64_t)n_workgroups * reps > (INT64_MAX / (kProbeThreads * 16))) return ROUTEPACK_E_INVALID;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    int rc = ROUTEPACK_E_DEVICE;
    float t = 0.f;
    if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) goto done;
    if (hipEventRecord(e0, stream) != hipSuccess) goto done;
    k_lds_read<<<n_workgroups, kProbeThreads, 0, stream>>>(reps, sink);
    if (hipGetLastError() != hipSuccess) goto done;
    if (hipEventRecord(e1, stream) != hipSuccess || hipEventSynchronize(e1) != hipSuccess) goto done;
    if (hipEventElapsedTime(&t, e0, e1) != hipSuccess) goto done;
    *ms = t;
    *bytes = (int64_t)n_workgroups * kProbeThreads * reps * 16;
    rc = ROUTEPACK_OK;
done:
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    return rc;
}
