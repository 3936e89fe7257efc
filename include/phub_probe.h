/*
 * phub_probe.h - bandwidth probe timed beside the exchange step.
 *
 * Measurement infrastructure, not part of the exchange step: read-only,
 * write-only and mixed read/write non-temporal streams over device buffers,
 * used to report measured HBM ceilings of the same buffers in the same run
 * as the step (the step's roofline is HBM bandwidth; the paper's section
 * 3.2.2 calls aggregation memory bound, and section 4.7 compares its
 * sustained bandwidth with a microbenchmark's ceiling).  Library:
 * libphub_probe.so.
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

/*
 * phub_probe_write - enqueue one write of `value` to elems_each floats of
 * each of nstreams device buffers (non-temporal stores), same launch shape
 * and argument rules as phub_probe_read.  The buffers are caller-owned and
 * overwritten.  Returns 0, -1 for invalid arguments (nothing launched), or
 * the HIP error code of the launch.
 */
int phub_probe_write(float *const *streams, int nstreams, int64_t elems_each, int grid,
                     float value, void *hip_stream);

/*
 * phub_probe_mixed - enqueue the exchange step's traffic without its
 * arithmetic: elems_each floats of each of the nread buffers read_streams
 * are read (as phub_probe_read), and elems_each floats of each of the nrw
 * buffers rw_streams are read and written back in place with the values
 * read (so their contents do not change), tile by tile, each tile written
 * back as soon as it is read.  1 <= nread + nrw <= 64; other arguments as
 * phub_probe_read.  Returns 0, -1 for invalid arguments (nothing launched),
 * or the HIP error code of the launch.
 */
int phub_probe_mixed(const float *const *read_streams, int nread, float *const *rw_streams,
                     int nrw, int64_t elems_each, int grid, float sentinel, float *sink,
                     void *hip_stream);

/* Elements per probe tile: elems_each must be a multiple of it. */
int phub_probe_tile_elems(void);

#ifdef __cplusplus
}
#endif

#endif /* PHUB_PROBE_H */
