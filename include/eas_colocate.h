/*
 * eas_colocate.h -- C ABI of the compute-unit reservation used to profile
 * encode under co-location (libeas.so).
 *
 * Paper Section 3.4 ("Dynamic SM partitioning"): the encode worker shares its
 * GPU with a local prefill worker on disjoint SM subsets, re-split every
 * micro-batch.  Encode latency is profiled at a few SM-allocation levels; a
 * level's table entry is the biggest batch size that runs nearly as fast there
 * as with the whole GPU, and at run time encode takes the smallest level whose
 * entry covers the current micro-batch.
 *
 * On MI355X the share is taken by occupancy: eas_cu_reserve launches n_cus
 * workgroups, each of which claims one whole compute unit (all of its LDS and
 * all of its vector registers), so kernels launched meanwhile run on the other
 * CUs only.  The workgroups are spread over the XCDs as the dispatcher places
 * them (round robin).  A held CU does no work.
 *
 * Conventions as in eas_encoder.h: every call returns an eas_status, argument
 * errors are found before anything is enqueued.
 */
#ifndef EAS_COLOCATE_H
#define EAS_COLOCATE_H

#include "eas_encoder.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Largest n_cus eas_cu_reserve accepts on a device of device_cus compute
 * units: all but one CU per shader engine (gfx950 has 8 CUs per shader
 * engine, so 224 of MI355X's 256).  Host only, no HIP calls; 0 for
 * device_cus <= 0. */
int32_t eas_cu_reserve_max(int32_t device_cus);

/* Holds n_cus compute units (1 <= n_cus <= eas_cu_reserve_max(CU count)) from the
 * moment the kernel enqueued on `stream` (hipStream_t as void*) starts until
 * *release != 0 or max_seconds (0 < max_seconds <= 60) have passed, whichever
 * comes first; every workgroup exits by the time limit at the latest.
 * started: host memory from hipHostMalloc, int32[n_cus], zeroed by the caller;
 *   workgroup b writes started[b] = 1 once it is resident, so the caller knows
 *   the share is held when all n_cus entries are 1.
 * release: host memory from hipHostMalloc, one int32, 0 at launch; the caller
 *   writes a non-zero value to end the reservation early.
 * Both stay allocated until the kernel has finished (synchronise `stream`).
 * Two limits of the occupancy form, found by measurement:
 *   - HIP maps streams onto a few hardware queues per process (4 by default),
 *     and streams sharing a queue run in order: work on a stream that shares
 *     `stream`'s queue waits for the reservation to end.  Keep the streams in
 *     use fewer than GPU_MAX_HW_QUEUES (set before HIP starts).
 *   - At least one CU per shader engine stays free (32 CUs on MI355X): with
 *     fewer, some shader engine has none, and other kernels stall behind it
 *     until the reservation ends; a larger n_cus is refused.
 * Returns EAS_ERR_INVALID_ARG for NULL pointers or out-of-range sizes, and
 * EAS_ERR_HIP if the launch fails. */
eas_status eas_cu_reserve(int32_t n_cus, double max_seconds, int32_t* started, const int32_t* release, void* stream);

#ifdef __cplusplus
}
#endif

#endif
