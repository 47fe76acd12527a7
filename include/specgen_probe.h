/*
 * specgen_probe.h -- memory-system ceilings on the current HIP device, for the
 * benchmark that reports the fork-decode kernels against them.  Separate
 * from the fork-decode library (libspecgen_probe.so): nothing here is part of
 * the attention, merge or block-move path.
 *
 * Both calls queue one kernel on `stream` and return 0, or a HIP error code
 * if the launch failed.  Buffers are device memory, 16-byte aligned, bytes a
 * multiple of 16 (else 1 = invalid argument, nothing queued).
 */
#ifndef SPECGEN_PROBE_H
#define SPECGEN_PROBE_H

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Reads `bytes` of src once, with 16-byte nontemporal vector loads spread over
 * every compute unit (contiguous chunks per workgroup).  sink: device uint32
 * written only if the data's xor has a value no test data produces (keeps the
 * loads alive). */
int specgen_probe_stream_read(const void *src, int64_t bytes, uint32_t *sink, hipStream_t stream);

/* Copies `bytes` from src to dst (not overlapping) with 16-byte nontemporal
 * vector loads and stores, batched eight per thread like the KV-block copies. */
int specgen_probe_stream_copy(void *dst, const void *src, int64_t bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* SPECGEN_PROBE_H */
