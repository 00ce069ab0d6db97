/*
 * routepack_probe.h -- measurement aid built beside the RoutePack library,
 * as its own shared library (libroutepack_probe.so); libroutepack.so does
 * not contain it.
 *
 * Not part of the method.  The annealing kernels keep each member's packing
 * state in LDS, so their roofline is quoted against the LDS read bandwidth
 * as well as HBM; this entry point measures that bandwidth on the device it
 * runs on, so the peak is a measured figure rather than a datasheet one.
 */
#ifndef ROUTEPACK_PROBE_H
#define ROUTEPACK_PROBE_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Streams reads through LDS at the full rate the device allows: a launch of
 * `n_workgroups` workgroups of 256 threads, each thread reading 16 bytes per
 * step for `reps` steps from a 64 KiB workgroup array, consecutive lanes on
 * consecutive 16-byte words (no bank conflicts).  What a thread reads is
 * folded into one word written to sink[workgroup * 256 + thread], so no read
 * is dead code.
 *   n_workgroups  >= 1; reps >= 1 (the bytes read must fit int64).
 *   sink          device uint32 [n_workgroups * 256], owned by the caller.
 *   ms            [host] out: duration of the launch from HIP events on
 *                 `stream`.
 *   bytes         [host] out: bytes read from LDS by the timed launch,
 *                 n_workgroups * 256 * reps * 16 (the fill of the array is
 *                 not counted).
 * Synchronizes.  Returns 0, ROUTEPACK_E_INVALID (-1) for a null pointer or a
 * size out of range, or ROUTEPACK_E_DEVICE (-6) for a HIP error.
 */
int routepack_probe_lds_read(int32_t n_workgroups, int32_t reps, uint32_t *sink, double *ms, int64_t *bytes,
                             hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* ROUTEPACK_PROBE_H */
