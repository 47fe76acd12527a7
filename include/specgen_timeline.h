/*
 * specgen_timeline.h -- per-workgroup timelines of the bf16 partial-attention
 * kernel (the MFMA partition's workers), for measuring where a launch spends
 * its time: start, plan copy, walk, the landing of every slot of the ring, end.
 *
 * Exported only by libspecgen_timeline.so: the fork-decode library (every
 * entry point of specgen.h, unchanged) with the partial kernel built under
 * SPECGEN_TIMELINE.  There, thread 0 of each workgroup reads the GPU's
 * constant 100 MHz clock (s_memrealtime) at those points into LDS, and the
 * workgroup writes the stamps to a device array when it ends; the slot loop
 * issues no extra memory operation.  libspecgen.so carries none of this.
 *
 * The array holds the stamps of the last launch that wrote each workgroup's
 * row (workgroups >= the recorded count are not recorded); rows of workgroups
 * a launch did not run keep what was there before, so clear it before a
 * launch whose rows are read.  All calls synchronise with the current device
 * and return 0, 1 (a null argument) or 2 (a HIP error).
 */
#ifndef SPECGEN_TIMELINE_H
#define SPECGEN_TIMELINE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Recorded workgroups and stamps per workgroup (the row length). */
int specgen_timeline_shape(int *workers, int *slots);

/* Copies the array to host memory: stamps (uint64 clock ticks of 10 ns, 0 =
 * not stamped) and kinds (int32), each workers x slots, row-major by
 * workgroup.  Slot 0: workgroup start (kind 100); 1: plan in LDS (101); 2:
 * walk done, block ids gathered (102); 3: the first three slots of the ring
 * issued (103; not stamped for a workgroup with no tiles); 4 + s: ring slot
 * s has landed and the
 * workgroup starts on it (kind -1 a q slot, 0 a prefix tile, 1 a suffix tile),
 * for the first slots - 5 slots; slots - 1: end (kind = the workgroup's slot
 * count). */
int specgen_timeline_read(uint64_t *stamps, int32_t *kinds);

/* Zeroes the array. */
int specgen_timeline_clear(void);

#ifdef __cplusplus
}
#endif
#endif /* SPECGEN_TIMELINE_H */
