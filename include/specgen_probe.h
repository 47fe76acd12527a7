/*
 * specgen_probe.h -- memory-system ceilings on the current HIP device, for the
 * benchmark that reports the fork-decode kernels against them.  Separate
 * from the fork-decode library (libspecgen_probe.so): nothing here is part of
 * the attention, merge or block-move path.
 *
 * Every call queues one kernel on `stream` and returns 0, or a HIP error
 * code if the launch failed.  Buffers are device memory; for the two plain
 * streams 16-byte aligned, bytes a multiple of 16 (else 1 = invalid
 * argument, nothing queued).
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

/* The bf16 partial-attention kernel's streaming pattern (head_dim 128) with
 * no arithmetic: `workers` workgroups of eight waves, each streaming an even
 * share of num_kv_heads * tiles_per_head tiles through four 32 KiB LDS stages
 * with LDS-DMA (three tiles in flight).  Tile k of kv head j moves, from each
 * of the pool blocks table[4k .. 4k + 3], head j's 4 KiB K slice of k_pool
 * and its 4 KiB V slice of v_pool: 32 KiB per tile, at the kernel's
 * granularity.  Pools: num_blocks blocks of num_kv_heads * 4 KiB each (the
 * library's pool layout at head_dim 128, bf16).  table: device int32, at least
 * 4 * tiles_per_head entries; ids are clamped into [0, num_blocks).  sink: as
 * above.  Returns 1 (nothing queued) for null or misaligned pointers,
 * non-positive sizes, or a share above 1024 tiles per workgroup. */
int specgen_probe_slice_ring(const void *k_pool, const void *v_pool, int64_t num_blocks, int num_kv_heads,
                             const int32_t *table, int tiles_per_head, int workers, uint32_t *sink,
                             hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* SPECGEN_PROBE_H */
