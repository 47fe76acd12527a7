/*
 * specgen_oracle.c -- plain fp64 CPU oracle for fork-decode attention, the
 * log-sum-exp merge, the KV-block import and export and the per-step append
 * of SpecGen (arXiv 2606.17518).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  The HIP library never
 * links, includes or calls it, and it includes nothing from the HIP side.
 *
 * What is computed, and where the paper fixes it:
 *   - Speculative forks are conditioned on the reasoning prefix and share its
 *     cached KV state; each fork then decodes over that shared prefix plus its
 *     own continuation (Sec. 1 "Introduction"; Sec. 4.2 "Insight: Speculative
 *     Generation"; Sec. 8.7 "Overhead", paragraph on prefix caching).
 *   - The remote prefix cache restores migrated KV state instead of
 *     recomputing the prefix from tokens (Sec. 6.2.3 "Remote Cache of
 *     Reasoning Prefixes").
 * The paper states no attention formula, no KV layout and no numeric format.
 * This oracle therefore takes the plain definition of single-query softmax
 * attention over the logically ordered keys (prefix tokens, then the fork's
 * own suffix tokens), evaluated in fp64, byte-for-byte block copies in both
 * directions, and an element copy of each fork's new token into the paged
 * layout.
 * The conventions it fixes where the paper is silent (GQA grouping, natural
 * log LSE, OCP E4M3 decode, a block-wide fp32 dequantisation scale, and the
 * paged layout: K pool [block][kv_head][slot][dim], V pool transposed as
 * [block][kv_head][dim][slot]) are listed with the header that declares the
 * GPU entry points.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ---- element decoding ---------------------------------------------------- */

/* bfloat16 is the upper half of an IEEE binary32; widening is exact. */
double specgen_ref_bf16_to_f64(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* OCP 8-bit floating point, E4M3 ("FN") variant, from the format definition:
 * 1 sign bit, 4 exponent bits with bias 7, 3 mantissa bits; exponent field 0
 * encodes subnormals m/8 * 2^-6; there are no infinities; S.1111.111 is NaN.
 * Largest finite magnitude: 1.75 * 2^8 = 448. */
double specgen_ref_e4m3_to_f64(uint8_t code) {
  int sign = (code >> 7) & 1;
  int e = (code >> 3) & 0xF;
  int m = code & 0x7;
  double v;
  if (e == 0xF && m == 0x7) return NAN;
  if (e == 0)
    v = ldexp((double)m / 8.0, -6);
  else
    v = ldexp(1.0 + (double)m / 8.0, e - 7);
  return sign ? -v : v;
}

void specgen_ref_decode_bf16(const uint16_t *src, int64_t n, double *dst) {
  for (int64_t i = 0; i < n; ++i) dst[i] = specgen_ref_bf16_to_f64(src[i]);
}

void specgen_ref_decode_e4m3(const uint8_t *src, int64_t n, double *dst) {
  for (int64_t i = 0; i < n; ++i) dst[i] = specgen_ref_e4m3_to_f64(src[i]);
}

/* ---- dense single-query softmax attention (the definition) --------------- */

/* o[d] = sum_i w_i V[i][d] / sum_i w_i with w_i = exp(s_i - m),
 * s_i = sm_scale * <q, K[i]>, m = max_i s_i; lse = m + ln(sum_i w_i).
 * With no keys the output is 0 and lse = -inf (an empty part). */
void specgen_ref_attend_dense(const double *q, const double *K, const double *V,
                              int64_t n, int32_t D, double sm_scale, double *o,
                              double *lse) {
  for (int32_t d = 0; d < D; ++d) o[d] = 0.0;
  if (n <= 0) {
    *lse = -INFINITY;
    return;
  }
  double *s = (double *)malloc((size_t)n * sizeof(double));
  double m = -INFINITY;
  for (int64_t i = 0; i < n; ++i) {
    double acc = 0.0;
    for (int32_t d = 0; d < D; ++d) acc += q[d] * K[i * D + d];
    s[i] = sm_scale * acc;
    if (s[i] > m) m = s[i];
  }
  double z = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    s[i] = exp(s[i] - m);
    z += s[i];
  }
  for (int64_t i = 0; i < n; ++i)
    for (int32_t d = 0; d < D; ++d) o[d] += s[i] * V[i * D + d];
  for (int32_t d = 0; d < D; ++d) o[d] /= z;
  *lse = m + log(z);
  free(s);
}

/* ---- fork-decode attention over a paged, shared-prefix KV cache ---------- */

typedef struct {
  int32_t num_traces, num_forks;     /* T, N = sum of forks over traces      */
  int32_t num_q_heads, num_kv_heads; /* Hq, Hkv (Hq a multiple of Hkv)        */
  int32_t head_dim, block_size;      /* D, tokens per KV block                */
  int64_t num_blocks;                /* pool capacity in blocks               */
  double sm_scale;
  int32_t kv_dtype;                  /* 0 = bf16, 1 = OCP E4M3 + block scale  */
  int32_t pad_;
  const uint16_t *q;                 /* [N][Hq][D] bf16 bits                  */
  const void *k_pool;                /* [num_blocks][Hkv][bs][D]              */
  const void *v_pool;                /* [num_blocks][Hkv][D][bs]              */
  const float *k_scale, *v_scale;    /* [num_blocks] (E4M3 only)              */
  const int32_t *fork_off;           /* [T+1]                                 */
  const int32_t *prefix_len;         /* [T]                                   */
  const int32_t *prefix_table_off;   /* [T+1]                                 */
  const int32_t *prefix_table;
  const int32_t *suffix_len;         /* [N]                                   */
  const int32_t *suffix_table_off;   /* [N+1]                                 */
  const int32_t *suffix_table;
  const int32_t *prefix_parent;      /* [T] parent trace or -1; NULL: all -1  */
} specgen_ref_batch_t;

/* Element d of kv head j of one cached token: slot `slot` of pool block blk.
 * Inside a block, head j's K is bs rows of D elements and its V is D rows of
 * bs elements. */
static double kv_elem(const specgen_ref_batch_t *b, int is_v, int64_t blk, int64_t slot, int32_t j,
                      int32_t d) {
  const int64_t D = b->head_dim, bs = b->block_size;
  const int64_t head = blk * b->num_kv_heads + j;
  const int64_t idx = is_v ? (head * D + d) * bs + slot : (head * bs + slot) * D + d;
  const void *pool = is_v ? b->v_pool : b->k_pool;
  if (b->kv_dtype == 0) return specgen_ref_bf16_to_f64(((const uint16_t *)pool)[idx]);
  const float *scale = is_v ? b->v_scale : b->k_scale;
  return specgen_ref_e4m3_to_f64(((const uint8_t *)pool)[idx]) * (double)scale[blk];
}

static int32_t trace_of_fork(const specgen_ref_batch_t *b, int32_t f) {
  for (int32_t t = 0; t < b->num_traces; ++t)
    if (f >= b->fork_off[t] && f < b->fork_off[t + 1]) return t;
  return -1;
}

/* The prefix a fork of trace t is conditioned on.  A fork taken at a later
 * trigger point of the same reasoning trace sees a longer prefix that extends
 * the one seen by earlier forks (Algorithm 1; Sec. 4.2): trace t's own
 * prefix tokens then continue its parent's whole prefix.  Writes the chain
 * root first into chain[] and returns its length (-1 on a cycle). */
static int32_t prefix_chain(const specgen_ref_batch_t *b, int32_t t, int32_t *chain) {
  int32_t n = 0;
  for (int32_t c = t; c >= 0; c = b->prefix_parent ? b->prefix_parent[c] : -1) {
    if (n == b->num_traces) return -1;
    chain[n++] = c;
  }
  for (int32_t i = 0; i < n / 2; ++i) {
    const int32_t x = chain[i];
    chain[i] = chain[n - 1 - i];
    chain[n - 1 - i] = x;
  }
  return n;
}

/* One output row (fork f, query head h): gather the fork's keys and values in
 * logical order (the prefix tokens of every trace on its chain, root first,
 * each in its own block table; then the fork's suffix tokens), then apply the
 * dense definition.  q head h reads kv head h / (Hq / Hkv). */
static void fork_row_upto(const specgen_ref_batch_t *b, int32_t f, int32_t h, int64_t suffix_keys,
                          const uint16_t *q_row, double *out_row, double *lse_out);

static void fork_row(const specgen_ref_batch_t *b, int32_t f, int32_t h,
                     double *out_row, double *lse_out) {
  fork_row_upto(b, f, h, b->suffix_len[f], b->q + ((int64_t)f * b->num_q_heads + h) * b->head_dim, out_row,
                lse_out);
}

/* The same with the fork's suffix cut to its first suffix_keys tokens and the
 * query given explicitly (one query of a multi-token prefill). */
static void fork_row_upto(const specgen_ref_batch_t *b, int32_t f, int32_t h, int64_t suffix_keys,
                          const uint16_t *q_row, double *out_row, double *lse_out) {
  const int32_t D = b->head_dim, bs = b->block_size;
  const int32_t g = b->num_q_heads / b->num_kv_heads;
  const int32_t j = h / g;
  int32_t chain[64];
  const int32_t L = prefix_chain(b, trace_of_fork(b, f), chain);
  int64_t n = suffix_keys;
  for (int32_t c = 0; c < L; ++c) n += b->prefix_len[chain[c]];
  double *q = (double *)malloc((size_t)D * sizeof(double));
  double *K = (double *)malloc((size_t)(n > 0 ? n : 1) * D * sizeof(double));
  double *V = (double *)malloc((size_t)(n > 0 ? n : 1) * D * sizeof(double));
  for (int32_t d = 0; d < D; ++d) q[d] = specgen_ref_bf16_to_f64(q_row[d]);
  int64_t i = 0;
  for (int32_t c = 0; c < L; ++c) {
    const int32_t t = chain[c];
    for (int64_t x = 0; x < b->prefix_len[t]; ++x, ++i) {
      const int64_t blk = b->prefix_table[b->prefix_table_off[t] + x / bs];
      for (int32_t d = 0; d < D; ++d) {
        K[i * D + d] = kv_elem(b, 0, blk, x % bs, j, d);
        V[i * D + d] = kv_elem(b, 1, blk, x % bs, j, d);
      }
    }
  }
  for (int64_t x = 0; x < suffix_keys; ++x, ++i) {
    const int64_t blk = b->suffix_table[b->suffix_table_off[f] + x / bs];
    for (int32_t d = 0; d < D; ++d) {
      K[i * D + d] = kv_elem(b, 0, blk, x % bs, j, d);
      V[i * D + d] = kv_elem(b, 1, blk, x % bs, j, d);
    }
  }
  specgen_ref_attend_dense(q, K, V, n, D, b->sm_scale, out_row, lse_out);
  free(q);
  free(K);
  free(V);
}

/* rows: nrows (fork, q head) pairs, or NULL for every row in (f, h) order.
 * out: [nrows][D] (or [N][Hq][D]); out_lse: [nrows] (or [N][Hq]).
 * Returns 0, or -1 if the batch is malformed. */
int specgen_ref_fork_decode_attn(const specgen_ref_batch_t *b, const int32_t *rows,
                                 int64_t nrows, double *out, double *out_lse,
                                 int32_t nthreads) {
  if (!b || b->num_kv_heads <= 0 || b->num_q_heads % b->num_kv_heads != 0) return -1;
  if (b->prefix_parent) {
    int32_t chain[64];
    if (b->num_traces > 64) return -1;
    for (int32_t t = 0; t < b->num_traces; ++t)
      if (b->prefix_parent[t] < -1 || b->prefix_parent[t] >= b->num_traces || prefix_chain(b, t, chain) < 0)
        return -1;
  }
  const int64_t total = rows ? nrows : (int64_t)b->num_forks * b->num_q_heads;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < total; ++r) {
    int32_t f, h;
    if (rows) {
      f = rows[2 * r];
      h = rows[2 * r + 1];
    } else {
      f = (int32_t)(r / b->num_q_heads);
      h = (int32_t)(r % b->num_q_heads);
    }
    fork_row(b, f, h, out + r * b->head_dim, out_lse + r);
  }
  return 0;
}

/* Multi-token prefill of every fork over its cached prefix: the speculative
 * prompt adds a few tokens per fork (a switch of the chat template to the
 * non-reasoning mode, Sec. 6.1.1 and Sec. 8.1) that are processed against the
 * cached reasoning prefix (Sec. 8.7, prefix caching paragraph).  Fork f's last
 * q_len[f] suffix tokens are queries: query i (0-based) sits at suffix
 * position S_f - q_len[f] + i and attends to the fork's whole prefix chain
 * and to suffix tokens 0 .. S_f - q_len[f] + i (causal inside the suffix).
 * b->q holds the queries [sum q_len][Hq][D], fork by fork.  rows: nrows
 * (query index, q head) pairs, or NULL for all.  Returns 0, or -1 if the
 * batch or q_len is malformed. */
int specgen_ref_fork_prefill_attn(const specgen_ref_batch_t *b, const int32_t *q_len, const int32_t *rows,
                                  int64_t nrows, double *out, double *out_lse, int32_t nthreads) {
  if (!b || !q_len || b->num_kv_heads <= 0 || b->num_q_heads % b->num_kv_heads != 0) return -1;
  int64_t nq = 0;
  for (int32_t f = 0; f < b->num_forks; ++f) {
    if (q_len[f] < 1 || q_len[f] > b->suffix_len[f]) return -1;
    nq += q_len[f];
  }
  int32_t *qf = (int32_t *)malloc((size_t)nq * sizeof(int32_t));   /* fork of each query */
  int64_t *qi = (int64_t *)malloc((size_t)nq * sizeof(int64_t));   /* its index in the fork */
  for (int32_t f = 0, k = 0; f < b->num_forks; ++f)
    for (int32_t i = 0; i < q_len[f]; ++i, ++k) {
      qf[k] = f;
      qi[k] = i;
    }
  const int64_t total = rows ? nrows : nq * b->num_q_heads;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < total; ++r) {
    int64_t v;
    int32_t h;
    if (rows) {
      v = rows[2 * r];
      h = rows[2 * r + 1];
    } else {
      v = r / b->num_q_heads;
      h = (int32_t)(r % b->num_q_heads);
    }
    const int32_t f = qf[v];
    const int64_t keys = (int64_t)b->suffix_len[f] - q_len[f] + qi[v] + 1;
    fork_row_upto(b, f, h, keys, b->q + (v * b->num_q_heads + h) * b->head_dim, out + r * b->head_dim,
                  out_lse + r);
  }
  free(qf);
  free(qi);
  return 0;
}

int32_t specgen_ref_max_threads(void) {
#ifdef _OPENMP
  return (int32_t)omp_get_max_threads();
#else
  return 1;
#endif
}

/* ---- log-sum-exp merge of partial results -------------------------------- */

/* o_parts [S][R][D] normalised partial outputs, lse_parts [S][R] natural-log
 * partial LSEs (-inf marks an empty part, whose o is ignored).  For each row:
 * M = max_s lse_s, w_s = exp(lse_s - M), out = sum_s w_s o_s / sum_s w_s,
 * lse = M + ln(sum_s w_s); a row whose parts are all empty gives out = 0 and
 * lse = -inf. */
void specgen_ref_lse_merge(const float *o_parts, const float *lse_parts, int32_t S,
                           int64_t R, int32_t D, double *out, double *out_lse) {
  for (int64_t r = 0; r < R; ++r) {
    double M = -INFINITY;
    for (int32_t s = 0; s < S; ++s) {
      const double l = lse_parts[(int64_t)s * R + r];
      if (l > M) M = l;
    }
    double *o = out + r * D;
    for (int32_t d = 0; d < D; ++d) o[d] = 0.0;
    if (M == -INFINITY) {
      out_lse[r] = -INFINITY;
      continue;
    }
    double z = 0.0;
    for (int32_t s = 0; s < S; ++s) {
      const double l = lse_parts[(int64_t)s * R + r];
      if (l == -INFINITY) continue;
      const double w = exp(l - M);
      z += w;
      const float *op = o_parts + ((int64_t)s * R + r) * D;
      for (int32_t d = 0; d < D; ++d) o[d] += w * (double)op[d];
    }
    for (int32_t d = 0; d < D; ++d) o[d] /= z;
    out_lse[r] = M + log(z);
  }
}

/* ---- KV-block import (restore) ------------------------------------------- */

/* Staging block i (block_bytes contiguous bytes at src + i*block_bytes) is
 * copied to pool block dst_ids[i]; ids outside [0, num_dst_blocks) are
 * skipped.  Returns the number of skipped ids. */
int64_t specgen_ref_kv_import(uint8_t *dst_pool, const uint8_t *src, int64_t block_bytes,
                              const int32_t *dst_ids, int64_t n, int64_t num_dst_blocks) {
  int64_t bad = 0;
  for (int64_t i = 0; i < n; ++i) {
    const int64_t id = dst_ids[i];
    if (id < 0 || id >= num_dst_blocks) {
      ++bad;
      continue;
    }
    memcpy(dst_pool + id * block_bytes, src + i * block_bytes, (size_t)block_bytes);
  }
  return bad;
}

/* ---- KV-block export (migration to the remote cache) --------------------- */

/* The direction opposite to the import: suspending a prefix moves its KV
 * state out of the serving cache into spare memory (Sec. 6.2.3).  Pool block
 * src_ids[i] is copied to staging block i; ids outside [0, num_src_blocks)
 * are skipped and leave staging block i as it was.  Returns the number of
 * skipped ids. */
int64_t specgen_ref_kv_export(uint8_t *staging, const uint8_t *pool, int64_t block_bytes,
                              const int32_t *src_ids, int64_t n, int64_t num_src_blocks) {
  int64_t bad = 0;
  for (int64_t i = 0; i < n; ++i) {
    const int64_t id = src_ids[i];
    if (id < 0 || id >= num_src_blocks) {
      ++bad;
      continue;
    }
    memcpy(staging + i * block_bytes, pool + id * block_bytes, (size_t)block_bytes);
  }
  return bad;
}

/* ---- Per-step append of each fork's new token ----------------------------- */

/* Every decode step of a fork adds one token to its private continuation,
 * whose KV is kept after the shared reasoning prefix (Sec. 4.2; Sec. 8.7,
 * prefix caching paragraph).  Fork f's new token takes logical suffix
 * position pos[f]: block suffix_table[suffix_table_off[f] + pos[f] / 16],
 * slot pos[f] % 16 (a position that is a multiple of 16 opens the next block
 * of the fork's table).  For kv head j and dim d, with element size es bytes:
 *   K pool byte offset ((b*Hkv + j)*16 + slot)*D + d   (times es)
 *   V pool byte offset ((b*Hkv + j)*D + d)*16 + slot   (times es)
 * receive k_new[f][j][d] and v_new[f][j][d].  A fork whose position has no
 * table entry, or whose block id lies outside [0, num_blocks), is skipped.
 * Returns the number of skipped forks. */
int64_t specgen_ref_kv_append(uint8_t *k_pool, uint8_t *v_pool, const uint8_t *k_new,
                              const uint8_t *v_new, int32_t es, int32_t N, int32_t Hkv, int32_t D,
                              const int32_t *pos, const int32_t *suffix_table_off,
                              const int32_t *suffix_table, int64_t num_blocks) {
  int64_t bad = 0;
  for (int32_t f = 0; f < N; ++f) {
    const int32_t p = pos[f];
    const int32_t nb = suffix_table_off[f + 1] - suffix_table_off[f];
    if (p < 0 || p / 16 >= nb) {
      ++bad;
      continue;
    }
    const int64_t b = suffix_table[suffix_table_off[f] + p / 16];
    if (b < 0 || b >= num_blocks) {
      ++bad;
      continue;
    }
    const int64_t slot = p % 16;
    for (int32_t j = 0; j < Hkv; ++j) {
      for (int32_t d = 0; d < D; ++d) {
        const int64_t src = ((int64_t)f * Hkv + j) * D + d;
        const int64_t ko = ((b * Hkv + j) * 16 + slot) * D + d;
        const int64_t vo = ((b * Hkv + j) * D + d) * 16 + slot;
        memcpy(k_pool + ko * es, k_new + src * es, (size_t)es);
        memcpy(v_pool + vo * es, v_new + src * es, (size_t)es);
      }
    }
  }
  return bad;
}
