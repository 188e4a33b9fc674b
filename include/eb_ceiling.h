/*
 * eb_ceiling.h -- attainable-bandwidth probe for the gather's roofline.
 *
 * Measurement only: it is not part of the pooled-lookup path (include/eb.h).
 * A gather of embedding rows (arXiv 2512.05831, Sec. 4.1 and the second
 * kernel of Sec. 4.3) reads one independent row per lookup, so its ceiling is
 * the rate at which the memory system serves random whole-row reads over the
 * tables' footprint, which lies below the streaming peak.  This probe reads
 * such rows with nothing else to do, giving that ceiling for a benchmark to
 * set the gather's achieved bandwidth against.
 */
#ifndef EB_CEILING_H
#define EB_CEILING_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * eb_probe_random_rows -- read rows ids[0..n) of a device table, each whole.
 *
 *   table           device memory of rows * row_bytes bytes, 16-byte aligned.
 *   rows            rows in the table, >= 1.
 *   row_bytes       32, 64, 128, 256, 512 or 1024.
 *   ids             device int32 [n]; every value must lie in [0, rows)
 *                   (not checked: the caller generates them in range).
 *   n               number of rows to read, >= 1.
 *   rows_in_flight  2, 4 or 8 rows per lane between waits.
 *   nontemporal     non-zero: non-temporal loads (bypassing L2 and the
 *                   last-level cache).
 *   grid            workgroups of 256 lanes, >= 1 (the loop strides over n).
 *   sink            device float [1]; written only in a case that does not
 *                   arise in practice (it keeps the loads live).
 *   stream          a hipStream_t; asynchronous.
 *
 * Returns 0; -1 for a bad argument, -2 for an unsupported row size, -3 when
 * the launch fails.  Allocates nothing.
 */
int eb_probe_random_rows(const void *table, int64_t rows, int32_t row_bytes, const int32_t *ids,
                         int64_t n, int32_t rows_in_flight, int32_t nontemporal, int32_t grid,
                         float *sink, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* EB_CEILING_H */
