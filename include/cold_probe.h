/* cold_probe.h -- a measurement aid that sits beside the scoring library
 * (libcold_probe.so, not libcold.so): the plainest gather of 32-byte table
 * rows, used to time the scattered row reads of a scoring call without the
 * work the gather does around them (the SE block of Section 3.2, the
 * reweighting, the user-side broadcast of Section 3.3).  It is not part of
 * the scoring path and computes no part of the model.
 *
 * Error behaviour: returns 0 after enqueueing the kernel, -1 for a null
 * pointer, a negative count or a table without rows (nothing is enqueued),
 * -2 if the launch fails. */
#ifndef COLD_PROBE_H
#define COLD_PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* out[i] = table[idx[i]] for i in [0, n): rows of 32 bytes.
 *   table       device, table_rows rows of 32 bytes, 16-byte aligned
 *   idx         device, n int64 row indices; an index outside
 *               [0, table_rows) reads row 0
 *   out         device, n rows of 32 bytes, 16-byte aligned, written
 *   stream      hipStream_t (NULL: the null stream); asynchronous
 * The caller owns every buffer. */
int cold_probe_row_gather(const void *table, int64_t table_rows, const int64_t *idx, void *out,
                          int64_t n, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* COLD_PROBE_H */
