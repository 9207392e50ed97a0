/*
 * dtree_probe.h -- measurement helpers of the tree-evaluator library.
 *
 * Not part of the evaluation method.  A plain streaming copy whose traffic is known
 * exactly: it calibrates hardware byte counters (FETCH_SIZE / WRITE_SIZE per dispatch)
 * and measures the HBM bandwidth a simple kernel reaches on the same device, next to
 * the datasheet peak.
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

#ifdef __cplusplus
}
#endif

#endif /* DTREE_PROBE_H */
