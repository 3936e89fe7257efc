/*
 * phub_probe.h - bandwidth probe timed beside the exchange step.
 *
 * Measurement infrastructure, not part of the exchange step: a read-only,
 * non-temporal stream over device buffers, used to report the measured HBM
 * read ceiling of the same buffers in the same run as the step (the step's
 * roofline is HBM bandwidth; the paper's section 3.2.2 calls aggregation
 * memory bound).  Library: libphub_probe.so.
 */
#ifndef PHUB_PROBE_H
#define PHUB_PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * phub_probe_read - enqueue one read of elems_each floats from each of
 * nstreams device buffers on hip_stream (a hipStream_t; NULL = the null
 * stream), with `grid` workgroups of 256 threads.
 *   streams    host array of nstreams device pointers (1..64), each
 *              16-byte aligned; caller-owned, read only.
 *   elems_each a multiple of phub_probe_tile_elems() (>= 0).
 *   sentinel   a lane stores its sum into sink only if it equals this value
 *              (keeps the loads alive; pass a value the data cannot sum to).
 *   sink       device buffer of grid * 256 floats, caller-owned.
 * Returns 0, -1 for invalid arguments (nothing launched), or the HIP error
 * code of the launch.  Timing is the caller's (events on hip_stream).
 */
int phub_probe_read(const float *const *streams, int nstreams, int64_t elems_each, int grid,
                    float sentinel, float *sink, void *hip_stream);

/* Elements per probe tile: elems_each must be a multiple of it. */
int phub_probe_tile_elems(void);

#ifdef __cplusplus
}
#endif

#endif /* PHUB_PROBE_H */
