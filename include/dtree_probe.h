/*
 * dtree_probe.h -- measurement helpers of the tree-evaluator library.
 *
 * Not part of the evaluation method.  A plain streaming copy and a plain streaming read
 * whose traffic is known exactly: they calibrate hardware byte counters (FETCH_SIZE /
 * WRITE_SIZE per dispatch) and measure the HBM bandwidth a simple kernel reaches on the
 * same device, next to the datasheet peak.
 */
#ifndef DTREE_PROBE_H
#define DTREE_PROBE_H

#include <stdint.h>

#include "dtree.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Copy `bytes` bytes from d_src to d_dst (device pointers, 16-byte aligned, bytes a
 * multiple of 16, buffers not overlapping) with one kernel launch on `stream`
 * (a hipStream_t; NULL = null stream).  Asynchronous.  Reads exactly `bytes` and writes
 * exactly `bytes`.
 * Errors: DT_ERR_INVALID_ARG (null pointer with bytes > 0, misalignment, bytes < 0 or not
 * a multiple of 16), DT_ERR_HIP (launch failure).
 */
dt_status dt_probe_copy(const void *d_src, void *d_dst, int64_t bytes, void *stream);

/*
 * Read `bytes` bytes from d_src (device pointer, 16-byte aligned, bytes a multiple of 16)
 * with one kernel launch of waves_per_cu wavefronts per compute unit (1..32), each reading
 * 16 KiB tiles with 16-byte non-temporal loads.  d_sink: a device int32 the kernel may
 * write (in practice it never does; it keeps the reads from being optimised away).
 * Asynchronous on `stream`.  The streaming-read ceiling the tree kernels are compared with.
 * Errors: DT_ERR_INVALID_ARG (null pointer with bytes > 0, misalignment, bytes < 0 or not
 * a multiple of 16, waves_per_cu out of range), DT_ERR_HIP (launch failure).
 */
dt_status dt_probe_read(const void *d_src, int64_t bytes, int32_t *d_sink, int32_t waves_per_cu,
                        void *stream);

#ifdef __cplusplus
}
#endif

#endif /* DTREE_PROBE_H */
