/*
 * specgen.h -- C ABI of the MI355X (gfx950) fork-decode attention, KV-block
 * import/export and per-step append library behind SpecGen's speculative generation
 * (arXiv 2606.17518).
 *
 * The paper forks non-reasoning generations off a long reasoning trace; every
 * fork is conditioned on the trace's prefix and reuses its cached KV state,
 * then continues with a short private suffix (Sec. 1; Sec. 4.2 "Insight:
 * Speculative Generation"; Sec. 8.7, prefix caching paragraph).  A fork event
 * launches K forks, K set from the resource capacity (Algorithm 1), and
 * idle-triggered forking adds more forks on the same prefix
 * (Sec. 6.1.1), so one trace's prefix is shared by F forks.  Successive
 * trigger points of one trace fork from ever longer prefixes while the
 * reasoning generation continues (Algorithm 1), so forks of different
 * trigger points share the earlier part: nested prefixes, stored once as a
 * chain of traces (prefix_parent_h).  Suspended
 * prefixes are kept in spare GPU memory and restored into the serving cache
 * instead of being recomputed (Sec. 6.2.3 "Remote Cache of Reasoning
 * Prefixes").
 *
 * Conventions fixed here (the paper states none of them):
 *  - Attention is single-query softmax attention with scale sm_scale > 0.
 *    For fork f of trace t and query head h the keys are, in logical order,
 *    the P_t prefix tokens of t followed by the S_f suffix tokens of f; the
 *    current decode token's own K/V is expected to be in the suffix already.
 *  - Grouped-query heads: q head h reads kv head h / (Hq / Hkv).
 *  - KV pools are paged in blocks of 16 tokens.  One block of one tensor is
 *    contiguous and holds Hkv head slices of 16*D elements each:
 *      K pool [num_blocks][Hkv][16][D]  (16 token rows of D values),
 *      V pool [num_blocks][Hkv][D][16]  (transposed: D rows of 16 tokens),
 *    i.e. K element (block b, kv head j, slot t, dim d) sits at
 *    ((b*Hkv + j)*16 + t)*D + d and the V element at ((b*Hkv + j)*D + d)*16 + t.
 *    A block table lists physical block ids in logical order; the last block
 *    of a prefix or suffix may be partly filled, and the values in its unused
 *    slots do not matter (they may be any bits, NaN included).  A fork's
 *    suffix starts at slot 0 of its own first block.
 *  - out is bf16 (round to nearest even from fp32); out_lse is the natural-log
 *    log-sum-exp of the scaled scores, fp32.
 *  - E4M3 KV is the OCP 8-bit "E4M3FN" format (bias 7, max 448, no inf,
 *    0x7F/0xFF NaN) with one fp32 scale per physical block and tensor: the
 *    value of a stored code c in block b is decode(c) * scale[b].  Scales are
 *    quantisation scales (e.g. the block's largest |value| / 448): finite and
 *    >= 0 (0: every value of the block is 0, as for an all-zero block); a
 *    negative scale gives unspecified results, and positive scales below
 *    2^-96 lose accuracy.
 *
 * Ownership: the caller allocates every buffer and keeps it alive until the
 * work queued on `stream` has finished.  The library keeps no pointer after a
 * call returns; host-side index mirrors are read only during the call.
 * Errors: every entry point returns a status; argument checks all run before
 * anything is queued, so SPECGEN_ERR_INVALID_ARG, SPECGEN_ERR_UNSUPPORTED
 * and SPECGEN_ERR_WORKSPACE mean nothing was launched and no output was
 * written.  SPECGEN_ERR_DEVICE (a failed launch) may leave the call's earlier
 * kernels queued: its outputs and workspace are then unspecified.
 * specgen_last_error() gives a message for the calling thread's most recent
 * non-OK status.
 * Streams: all work is asynchronous on `stream` (0 = the null stream) of the
 * current HIP device.  Results are deterministic: the work split depends only
 * on the lengths, and no floating-point atomics are used.  A call queues
 * kernel launches only (no allocation, copy or memset), so it can be captured
 * into a HIP graph; a replay uses the lengths of the captured call and the
 * device buffers' contents at replay time.
 */
#ifndef SPECGEN_H
#define SPECGEN_H

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SPECGEN_OK = 0,
  SPECGEN_ERR_INVALID_ARG = 1, /* a null pointer, size or shape out of range */
  SPECGEN_ERR_UNSUPPORTED = 2, /* a valid request the library does not serve */
  SPECGEN_ERR_WORKSPACE = 3,   /* workspace missing or too small            */
  SPECGEN_ERR_DEVICE = 4       /* a HIP call or kernel launch failed        */
} specgen_status_t;

typedef enum { SPECGEN_BF16 = 0, SPECGEN_FP8_E4M3 = 1, SPECGEN_FP32 = 2 } specgen_dtype_t;

/* Which kernel serves each work item.  AUTO: a prefix item uses the bf16 MFMA
 * kernel when its row count F_t * (Hq/Hkv) is at least 16 (F_t: the forks of
 * trace t and of every trace nested below it), else the
 * wavefront dot kernel; suffix items use the MFMA kernel.  DOT / MFMA force
 * one kernel for every item (used by tests to cover both paths). */
typedef enum { SPECGEN_PATH_AUTO = 0, SPECGEN_PATH_DOT = 1, SPECGEN_PATH_MFMA = 2 } specgen_path_t;

/* Options of a fork batch (the flags field).
 * SPECGEN_FLAG_FP8_SCORES: with E4M3 KV and head_dim 128, the MFMA kernel
 * computes the scores q . k on the fp8 matrix cores straight from the K codes
 * (no decode of K), with each query row held as two E4M3 terms,
 * q = 2^e (hi + lo/16), e from the row's largest |q|: the scores stay within
 * the accuracy of bf16 queries.  Values and probabilities stay bf16.  Items
 * on the dot path are unaffected.  With bf16 KV the flag is rejected
 * (SPECGEN_ERR_INVALID_ARG); with head_dim 64, SPECGEN_ERR_UNSUPPORTED.
 * Other bits must be 0. */
#define SPECGEN_FLAG_FP8_SCORES 1

/* One decode step for every fork of T traces. */
typedef struct {
  int32_t num_traces;        /* 1 <= T <= 32 per call                            */
  int32_t num_forks;         /* N = sum_t F_t, 1 <= N <= 512 per call; forks are
                                grouped by trace.  Larger batches are
                                SPECGEN_ERR_UNSUPPORTED: split them over calls */
  int32_t num_q_heads;       /* Hq >= 1                                          */
  int32_t num_kv_heads;      /* Hkv >= 1, Hq % Hkv == 0, Hq / Hkv <= 128         */
  int32_t head_dim;          /* D: 64 or 128                                     */
  int32_t block_size;        /* must be 16                                       */
  int64_t num_blocks;        /* pool capacity in blocks (>= 1)                   */
  float sm_scale;            /* > 0 and finite, e.g. 1/sqrt(D)                   */
  int32_t kv_dtype;          /* specgen_dtype_t: SPECGEN_BF16 or SPECGEN_FP8_E4M3 */
  int32_t path;              /* specgen_path_t                                   */
  int32_t flags;             /* 0, or SPECGEN_FLAG_FP8_SCORES                    */
  /* device memory, caller-owned */
  const void *q;             /* [N][Hq][D] bf16                                  */
  const void *k_pool;        /* [num_blocks][Hkv][16][D] kv_dtype                */
  const void *v_pool;        /* [num_blocks][Hkv][D][16] kv_dtype (transposed)   */
  const float *k_scale;      /* [num_blocks] fp32 for E4M3, else NULL            */
  const float *v_scale;      /* [num_blocks] fp32 for E4M3, else NULL            */
  const int32_t *fork_off;   /* [T+1], fork_off[0] = 0, nondecreasing, [T] = N;
                                forks of trace t are [fork_off[t], fork_off[t+1]);
                                a trace has at least one fork of its own or in a
                                trace nested below it (prefix_parent_h)          */
  const int32_t *prefix_len; /* [T], P_t >= 1                                    */
  const int32_t *prefix_table_off; /* [T+1]; trace t's ids are
                                prefix_table[prefix_table_off[t] ..], at least
                                ceil(P_t/16) of them                            */
  const int32_t *prefix_table;
  const int32_t *suffix_len; /* [N], S_f >= 0                                    */
  const int32_t *suffix_table_off; /* [N+1], at least ceil(S_f/16) ids per fork  */
  const int32_t *suffix_table;     /* may be NULL only if every S_f is 0         */
  /* host mirrors of the index arrays above (same contents), read only during
     the call: they size the work split and the workspace and travel to the
     kernels with the launch; the block tables themselves are read on the
     device.  Mirrors and device arrays must agree. */
  const int32_t *fork_off_h;
  const int32_t *prefix_len_h;
  const int32_t *suffix_len_h;
  const int32_t *prefix_table_off_h;
  const int32_t *suffix_table_off_h;
  /* Nested prefixes (a fork tree), host only, read during the call: [T]
     parent trace of each trace, or -1 for a root; NULL makes every trace a
     root.  A fork of trace t attends over the prefix tokens of every trace
     on the chain root, ..., parent, t (in that order, each with its own
     block table and P), then its suffix.  Parents come first and traces are
     in depth-first order: prefix_parent_h[t] is t-1 or an ancestor of t-1.
     At most 8 traces on a chain.                                              */
  const int32_t *prefix_parent_h;
} specgen_fork_batch_t;

/* Workspace bytes that specgen_fork_decode_attn needs for this batch (partial
 * outputs of the split key axis).  Validates the batch like the call itself. */
specgen_status_t specgen_fork_decode_attn_workspace_size(const specgen_fork_batch_t *b,
                                                         size_t *bytes);

/* Fork-decode attention, one decode token per fork:
 *   out[f][h][:] = softmax(sm_scale * q[f][h] . K_seq^T) V_seq,
 *   out_lse[f][h] = ln sum_i exp(sm_scale * q[f][h] . K_seq[i])
 * where K_seq/V_seq are the prefix tokens of fork f's trace followed by f's
 * suffix tokens (kv head h / (Hq/Hkv)).  The shared prefix of each trace is
 * streamed from HBM once per kv head for all of the trace's forks and query
 * heads of a GQA group; each fork's suffix is streamed once.  The key axis is
 * split across workgroups and the partial results are merged with the
 * log-sum-exp rule (specgen_lse_merge computes the same merge standalone).
 *   out: [N][Hq][D] bf16, device.  out_lse: [N][Hq] fp32 device, or NULL.
 *   workspace: device, at least specgen_fork_decode_attn_workspace_size bytes,
 *   256-byte aligned; its contents on entry do not matter.
 * Block ids must lie in [0, num_blocks); an out-of-range id is undefined
 * behaviour (the kernels do not check it).  The library built with
 * SPECGEN_DEBUG_CHECKS defined (libspecgen_debug.so) checks every id the call
 * will read before anything is launched -- ceil(P_t/16) entries per trace and
 * ceil(S_f/16) per fork -- by copying the read part of each block table to
 * the host and synchronising `stream`; an id out of range returns
 * SPECGEN_ERR_INVALID_ARG naming the table entry.  That build is for testing:
 * its calls block and copy, so they cannot be captured into a graph.  The same
 * check guards specgen_fork_decode_attn_phase (PARTIALS and ALL),
 * specgen_fork_decode_attn_noalloc and specgen_fork_prefill_attn there. */
specgen_status_t specgen_fork_decode_attn(const specgen_fork_batch_t *b, void *out, float *out_lse,
                                          void *workspace, size_t workspace_bytes,
                                          hipStream_t stream);

/* specgen_fork_decode_attn for callers that cannot allocate device memory:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  It takes no workspace: the partial results live in a scratch
 * array of the library, SPECGEN_NOALLOC_SCRATCH_BYTES of device memory per
 * GPU, which each GPU the library runs on holds from the first call there
 * until the process ends.  The call allocates nothing.
 *   Arguments, results and errors as for specgen_fork_decode_attn; a batch
 *   whose workspace (specgen_fork_decode_attn_workspace_size) exceeds the
 *   scratch is rejected with SPECGEN_ERR_WORKSPACE before anything is queued.
 * All calls on one GPU share its scratch, which keeps the last call's
 * contents (none of which a later call reads: nothing needs clearing).  Calls
 * that overlap on one GPU -- on different streams, or from threads without
 * ordering -- race on it and give undefined results; calls ordered on one
 * stream are safe. */
#define SPECGEN_NOALLOC_SCRATCH_BYTES (64ull << 20)
specgen_status_t specgen_fork_decode_attn_noalloc(const specgen_fork_batch_t *b, void *out, float *out_lse,
                                                  hipStream_t stream);

/* How specgen_fork_decode_attn splits the key axis of a batch, for callers
 * that analyse load balance or place test inputs relative to the split.  Host
 * only: it runs the same planner as the call (on the current device's compute
 * unit count, 256 where no device is present) and launches nothing.  One
 * segment per (work item, workgroup) pair: the keys [first_token, first_token
 * + num_tokens) of the item that one workgroup processes and leaves as one
 * partial result.  A prefix item is (trace, kv head, row block) over the
 * trace's own P_t prefix tokens (token 0 = the trace's first own token); a
 * suffix item is (fork, kv head, row block) over the fork's S_f suffix tokens.
 *   b: as for the call; its device pointers are not read and may be NULL.
 *   segs: host array of cap entries (may be NULL when cap is 0); *count
 *   receives the number of segments, which may exceed cap (then only cap are
 *   written).  Validates the host mirrors like the call itself. */
typedef struct {
  int32_t kind;         /* 0: prefix item, 1: suffix item                      */
  int32_t trace;        /* trace of a prefix item; the fork's trace otherwise  */
  int32_t fork;         /* fork of a suffix item, -1 for a prefix item        */
  int32_t kv_head;
  int32_t row_block;    /* row block of the item                               */
  int32_t first_row;    /* the item's rows: [first_row, first_row + num_rows)
                           of its trace's rows (fork f - fork_off[t], q head
                           h % (Hq/Hkv) is row (f - fork_off[t]) * (Hq/Hkv)
                           + h % (Hq/Hkv)) for a prefix item, of the group's
                           q heads for a suffix item                          */
  int32_t num_rows;
  int32_t kernel;       /* 0: MFMA kernel, 1: dot kernel                       */
  int32_t worker;       /* workgroup index in that kernel's launch             */
  int32_t first_token;  /* first key of the segment within the item's keys    */
  int32_t num_tokens;   /* keys in the segment                                 */
} specgen_split_segment_t;
specgen_status_t specgen_fork_decode_attn_split(const specgen_fork_batch_t *b, specgen_split_segment_t *segs,
                                                int64_t cap, int64_t *count);

/* The two phases of specgen_fork_decode_attn, for callers that want to place
 * work or timing events between them.  SPECGEN_PHASE_PARTIALS runs the split
 * attention kernels, which leave one partial (o, lse) per worker and item in
 * the workspace; SPECGEN_PHASE_MERGE combines those partials into out and
 * out_lse.  PARTIALS followed by MERGE on the same stream, with the same batch
 * and workspace, gives exactly the result of one specgen_fork_decode_attn
 * call (SPECGEN_PHASE_ALL).  Arguments as for specgen_fork_decode_attn; `out`
 * may be NULL for PARTIALS. */
typedef enum { SPECGEN_PHASE_ALL = 0, SPECGEN_PHASE_PARTIALS = 1, SPECGEN_PHASE_MERGE = 2 } specgen_phase_t;
specgen_status_t specgen_fork_decode_attn_phase(const specgen_fork_batch_t *b, int32_t phase, void *out,
                                                float *out_lse, void *workspace, size_t workspace_bytes,
                                                hipStream_t stream);

/* Multi-token prefill of every fork over its cached prefix: the speculative
 * prompt appends a few tokens per fork (the chat template's switch to the
 * non-reasoning mode, Sec. 6.1.1 and Sec. 8.1) that are processed against the
 * cached reasoning prefix instead of recomputing it (Sec. 8.7, prefix caching
 * paragraph).  Fork f's last q_len_h[f] suffix tokens are queries (their K/V
 * already in the suffix, S_f counting them): query i (0-based) attends to
 * every prefix token of its chain and to suffix tokens 0 .. S_f - q_len_h[f]
 * + i (causal inside the suffix, one query row per (query, q head)).
 *   b: a fork batch as for specgen_fork_decode_attn, except that q is
 *      [Q][Hq][D] bf16 with Q = sum_f q_len_h[f], fork by fork in query order.
 *   q_len_h: host int32 [N], 1 <= q_len_h[f] <= S_f, read during the call;
 *      Q <= 512 per call.
 *   out: [Q][Hq][D] bf16; out_lse: [Q][Hq] fp32 or NULL.
 *   workspace: at least specgen_fork_prefill_attn_workspace_size bytes.
 * The work runs as a decode batch in which each query is a fork of its own
 * (same trace, same block table, its causal suffix length), so the shared
 * prefix is still read once per row block of 256 query rows per kv head. */
specgen_status_t specgen_fork_prefill_attn_workspace_size(const specgen_fork_batch_t *b, const int32_t *q_len_h,
                                                          size_t *bytes);
specgen_status_t specgen_fork_prefill_attn(const specgen_fork_batch_t *b, const int32_t *q_len_h, void *out,
                                           float *out_lse, void *workspace, size_t workspace_bytes,
                                           hipStream_t stream);

/* One tensor of a KV-block import: dst_pool is [num_dst_blocks][block_bytes],
 * src_staging is [n][block_bytes] contiguous (the restored remote copy). */
typedef struct {
  void *dst_pool;
  const void *src_staging;
  int64_t block_bytes;       /* > 0 and a multiple of 4; multiples of 16 take the
                                16-byte vector path                             */
} specgen_kv_tensor_t;

/* KV-block import (restore of a cached prefix, Sec. 6.2.3): for every tensor
 * and every i < n, copy staging block i to pool block dst_block_ids[i], byte
 * for byte.  Ids outside [0, num_dst_blocks) are skipped and, if
 * bad_id_count is not NULL, counted there (device int32, incremented, not
 * reset).  Destinations must be distinct; with duplicates the winner is
 * unspecified.  Staging and pool must not overlap.
 *   tensors: host array of 1..4 descriptors (e.g. K, V, K scales, V scales).
 *   dst_block_ids: device int32 [n].  n >= 0 (0 queues nothing). */
specgen_status_t specgen_kv_import(const specgen_kv_tensor_t *tensors, int32_t num_tensors,
                                   const int32_t *dst_block_ids, int64_t n,
                                   int64_t num_dst_blocks, int32_t *bad_id_count,
                                   hipStream_t stream);

/* One tensor of a KV-block export: src_pool is [num_src_blocks][block_bytes],
 * dst_staging is [n][block_bytes] contiguous (the copy a remote cache keeps). */
typedef struct {
  void *dst_staging;
  const void *src_pool;
  int64_t block_bytes;       /* as for specgen_kv_tensor_t                      */
} specgen_kv_export_tensor_t;

/* KV-block export (migration of a suspended prefix out of the serving cache,
 * Sec. 6.2.3; the reverse of specgen_kv_import): for every tensor and every
 * i < n, copy pool block src_block_ids[i] to staging block i, byte for byte.
 * Ids outside [0, num_src_blocks) are skipped (staging block i keeps its
 * bytes) and, if bad_id_count is not NULL, counted there (device int32,
 * incremented, not reset).  Repeated source ids are allowed.  Staging and
 * pool must not overlap.
 *   tensors: host array of 1..4 descriptors.
 *   src_block_ids: device int32 [n].  n >= 0 (0 queues nothing). */
specgen_status_t specgen_kv_export(const specgen_kv_export_tensor_t *tensors, int32_t num_tensors,
                                   const int32_t *src_block_ids, int64_t n,
                                   int64_t num_src_blocks, int32_t *bad_id_count,
                                   hipStream_t stream);

/* One decode step's new K/V token for each of N forks. */
typedef struct {
  int32_t num_forks;         /* N >= 0 (0 queues nothing)                        */
  int32_t num_kv_heads;      /* Hkv >= 1                                         */
  int32_t head_dim;          /* D: 1..1024                                       */
  int32_t kv_dtype;          /* SPECGEN_BF16 or SPECGEN_FP8_E4M3 (element size
                                2 or 1 byte; elements are copied as bits)        */
  int64_t num_blocks;        /* pool capacity in blocks (>= 1)                   */
  /* device memory, caller-owned */
  void *k_pool;              /* [num_blocks][Hkv][16][D]                         */
  void *v_pool;              /* [num_blocks][Hkv][D][16] (transposed)            */
  const void *k_new;         /* [N][Hkv][D], the new token's K per kv head       */
  const void *v_new;         /* [N][Hkv][D]                                      */
  const int32_t *pos;        /* [N], the suffix position each token takes: the
                                fork's suffix length before this step            */
  const int32_t *suffix_table_off; /* [N+1], nondecreasing                       */
  const int32_t *suffix_table;     /* fork f's ids are
                                suffix_table[suffix_table_off[f] ..
                                suffix_table_off[f+1]) in logical order          */
  int32_t *bad_count;        /* device int32 or NULL: forks skipped              */
} specgen_kv_append_t;

/* Per-step append (each fork's continuation grows by one token per decode
 * step after the shared prefix, Sec. 4.2; Sec. 8.7, prefix caching
 * paragraph): for every fork f, kv head j and dim d,
 *   b = suffix_table[suffix_table_off[f] + pos[f]/16], t = pos[f] % 16,
 *   K element (b, j, t, d) = k_new[f][j][d],  V element (b, j, d, t) = v_new[f][j][d]
 * in the layout of the fork batch.  A position that is a multiple of 16 opens
 * a fresh block: the caller lists it at the end of the fork's table first
 * (block allocation is the caller's).  A fork with pos < 0, with no table
 * entry for pos/16, or whose block id lies outside [0, num_blocks) is skipped
 * and, if bad_count is not NULL, counted (incremented, not reset).  Only the
 * listed elements are written.  E4M3 elements are copied as codes: they must
 * already be encoded with the target block's scale, which the caller owns and
 * sets for a fresh block.  Two forks writing the same (block, slot) race.
 * After the call, a fork batch with S_f = pos[f] + 1 attends over the new
 * token. */
specgen_status_t specgen_kv_append(const specgen_kv_append_t *a, hipStream_t stream);

/* Log-sum-exp merge of S partial attention results over disjoint key sets.
 * No passage of the paper defines this step: it serves through an inference
 * engine and gives no attention arithmetic.  The merge is the identity that
 * softmax attention over a union of disjoint key sets satisfies, which lets
 * the key axis of the fork-decode step (the shared prefix of Sec. 4.2 and
 * Sec. 8.7 plus each fork's suffix) be split across workgroups; the same
 * identity is how partial results from several devices would be combined.
 *   M = max_s lse[s][r]; w_s = exp(lse[s][r] - M);
 *   out[r] = sum_s w_s o[s][r] / sum_s w_s; out_lse[r] = M + ln sum_s w_s.
 * A part with lse = -inf is empty and its o is ignored; a row with only empty
 * parts gives out = 0 and out_lse = -inf.
 *   o_parts: device fp32 [S][R][D]; lse_parts: device fp32 [S][R] (natural log).
 *   out: device [R][D] of out_dtype (SPECGEN_BF16 or SPECGEN_FP32).
 *   out_lse: device fp32 [R] or NULL.  1 <= S, 0 <= R, 1 <= D <= 1024. */
specgen_status_t specgen_lse_merge(const float *o_parts, const float *lse_parts, int32_t num_parts,
                                   int64_t rows, int32_t head_dim, void *out, int32_t out_dtype,
                                   float *out_lse, hipStream_t stream);

/* Message for the calling thread's most recent non-OK status ("" if none). */
const char *specgen_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SPECGEN_H */
