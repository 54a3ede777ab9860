/* libkvgov_peaks: measured-peak microbenchmarks for MI355X (gfx950).
 *
 * Not part of the KVGov path.  The measurement harness reports each kernel of
 * the path against the chip's published peaks and also against what these two
 * kernels reach on the same device:
 *
 *   kvgov_peak_valu    32-bit integer vector throughput (rotate, 3-input add,
 *                      3-input xor: the op mix of a SHA-256 round), eight
 *                      independent dependency chains per lane;
 *   kvgov_peak_gather  HBM bandwidth of 32-byte reads at pseudo-random slots of
 *                      a table (the access pattern of a hash-table probe).
 *
 * Both are asynchronous on `stream` (a hipStream_t, NULL = default stream);
 * the caller times them with events on that stream.  All pointers are device
 * pointers owned by the caller.  Return 0, or a negative code below before
 * anything is enqueued.
 */
#ifndef KVGOV_PEAKS_H
#define KVGOV_PEAKS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KVGOV_PEAK_E_INVAL (-1) /* null pointer, non-positive size, bad table */
#define KVGOV_PEAK_E_HIP (-7)   /* the launch failed */

/* Launches `grid` workgroups of 256 lanes; each lane runs `trips` trips of
 * 4 x 8 x 3 integer ops and writes one word to out[lane] (out holds
 * grid*256 uint32).  *ops (host) receives the op count of the launch. */
int kvgov_peak_valu(uint32_t *out, int32_t grid, int32_t trips, int64_t *ops, void *stream);

/* Launches `grid` workgroups of 256 lanes; each lane reads `trips` x 4 records
 * of 32 bytes at pseudo-random slots of `table` (slots x 32 bytes, slots a
 * power of two <= 2^32, 16-byte aligned) and writes one word to out[lane].
 * *bytes (host) receives the bytes read by the launch. */
int kvgov_peak_gather(const uint8_t *table, int64_t slots, uint32_t *out, int32_t grid,
                      int32_t trips, int64_t *bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* KVGOV_PEAKS_H */
