/* semkv_timeline.h -- the one extra entry point of the tracing build of the
 * decode kernel (libsemkv_timeline.so, built by
 * `python paper_2608_28911_amd/build.py --timeline`).  The product library
 * libsemkv.so does not export it.
 *
 * In the tracing build, lane 0 of every wave of the first 4096 workgroups of
 * each decode launch writes the constant 100 MHz device clock at the end of
 * each phase of the kernel into a device array; a later launch overwrites it.
 * Layout: uint64 [4096 workgroups][16 waves][32 events], workgroup index
 * x + X (y + Y z) of the launch grid (X, Y its x and y extents), events:
 *   0 start, 1 tables and query operands built, 2 first record in LDS,
 *   3..7 the wave's 1st..5th record done with the next record's data in LDS
 *   (later records overwrite 7), 8 the first record's arithmetic done,
 *   9 the wave's records done,
 *   10 workgroup partial merged, 11 partial stored, 12 split counter taken,
 *   13 the last workgroup's merge done; slots 14 and 15 count the wave's
 *   value-sum flushes and records; 16..18 inside the wave's first record:
 *   the next record's loads issued, scores done, softmax and flush done;
 *   19..21 in the prologue: tables written, query value in hand, query runs
 *   done (16..21 only in the fine build, `build.py --timeline-fine`: they
 *   delay the paths they measure).
 * Slots a launch did not write keep their previous contents (zero at load).
 */
#ifndef SEMKV_TIMELINE_H
#define SEMKV_TIMELINE_H
#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Copy the stamp array to host memory `host` (caller-owned, `bytes` =
 * 4096 * 16 * 32 * 8).  Synchronous with respect to the device (waits for
 * prior work).  SEMKV_EINVAL on a null pointer or another size, SEMKV_EHIP
 * when the copy fails. */
int semkv_timeline_read(void* host, size_t bytes);

#ifdef __cplusplus
}
#endif
#endif
