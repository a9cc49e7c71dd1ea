/*
 * gba_ceilings.h -- measurement kernels beside the GBA push-step (libgba.so).
 *
 * Each call runs the simplest kernel that has one of the access patterns the
 * push-step is built from, so that the step's kernels can be judged against
 * what the memory system delivers for that pattern on this GPU:
 *   - a stream of 16-byte non-temporal reads (the dense weighted sum of
 *     Alg. 2 reads the K buffered gradients this way);
 *   - a stream copy, reads and writes of 16 bytes (known bytes both ways, for
 *     calibrating hardware byte counters);
 *   - gathers of whole table rows at random positions (the embedding row
 *     passes read the contribution rows, and the table rows, this way).
 * None of them is part of the step.  Conventions as in gba.h: device
 * pointers owned by the caller, work only enqueued on `stream`, host-visible
 * misuse returns a non-zero gba_status and enqueues nothing.
 */
#ifndef GBA_CEILINGS_H
#define GBA_CEILINGS_H

#include "gba.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Reads n16 16-byte vectors of src once, with non-temporal loads.
 *   src     [n16 * 16] bytes, 16-byte aligned; any contents.
 *   sink    [gba_ceiling_sink_words(blocks)] uint32 out: one word per wave
 *           (an XOR of what the wave read, so the loads are not removed).
 *   blocks  workgroups of 256 threads (>= 1); each takes 4 vectors per thread
 *           per round and walks the array in a grid-stride loop.
 * Bytes moved: 16 * n16 read, 4 per wave written.
 */
gba_status gba_ceiling_read(const void* src, int64_t n16, uint32_t* sink, int32_t blocks, hipStream_t stream);

/*
 * Copies n16 16-byte vectors from src to dst (non-temporal loads and stores).
 *   src, dst  [n16 * 16] bytes each, 16-byte aligned, not overlapping.
 *   blocks    workgroups of 256 threads (>= 1); each takes 8 vectors per
 *             thread per round and walks the arrays in a grid-stride loop.
 * Bytes moved: 16 * n16 read, 16 * n16 written.
 */
gba_status gba_ceiling_copy(const void* src, void* dst, int64_t n16, int32_t blocks, hipStream_t stream);

/*
 * Gathers n rows of D floats, table[rows[i]], in the order given, as the
 * embedding row passes do: D/4 lanes take one row (16 bytes each), and each
 * lane group has 8 rows in flight.
 *   table   [R][D] float, 16-byte aligned.
 *   rows    [n] int64 row numbers; one outside [0, R) is skipped.
 *   sink    [gba_ceiling_sink_words(blocks)] uint32 out, one word per wave.
 *   D % 4 == 0, 4 <= D <= GBA_MAX_D.
 * Bytes moved: n * D * 4 gathered, n * 8 of row numbers read.
 */
gba_status gba_ceiling_gather_rows(const float* table, int64_t R, int32_t D, const int64_t* rows, int64_t n,
                                   uint32_t* sink, int32_t blocks, hipStream_t stream);

/* Words of `sink` a call with this many blocks writes (one per wave). */
int64_t gba_ceiling_sink_words(int32_t blocks);

#ifdef __cplusplus
}
#endif
#endif /* GBA_CEILINGS_H */
