/* sanitize_driver.c -- drives every entry point of the fp64 oracle on small
 * random inputs whose buffers are allocated to their exact sizes, so that a
 * build with AddressSanitizer and UndefinedBehaviorSanitizer reports any
 * out-of-bounds access, leak or undefined operation in the oracle.  Compiled
 * and run on the CPU by tests/test_sanitizers.py (no GPU involved); it checks
 * a few results for sanity but its point is the sanitizer run. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../oracle/specgen_oracle.c"

static uint64_t rs = 0x9E3779B97F4A7C15ull;
static uint32_t rnd(void) {   /* xorshift64* */
  rs ^= rs >> 12;
  rs ^= rs << 25;
  rs ^= rs >> 27;
  return (uint32_t)((rs * 2685821657736338717ull) >> 32);
}
static double unif(void) { return (rnd() + 0.5) / 4294967296.0; }

static uint16_t bf16_of(double x) {   /* truncation is enough for test data */
  float f = (float)x;
  uint32_t u;
  memcpy(&u, &f, 4);
  return (uint16_t)(u >> 16);
}

static void *xmalloc(size_t n) {
  void *p = malloc(n ? n : 1);
  if (!p) abort();
  return p;
}

#define FAIL(...)                   \
  do {                              \
    fprintf(stderr, __VA_ARGS__);   \
    fprintf(stderr, "\n");          \
    exit(1);                        \
  } while (0)

/* One random fork batch: T traces (nested as a chain when `chain`), forks per
 * trace 1..3, prefix 1..40 tokens, suffix 0..33, every id distinct. */
static void run_batch(int T, int chain, int fp8, int Hq, int Hkv, int D) {
  int32_t *fork_off = xmalloc(sizeof(int32_t) * (T + 1));
  int32_t *plen = xmalloc(sizeof(int32_t) * T);
  int32_t *ptoff = xmalloc(sizeof(int32_t) * (T + 1));
  int32_t *parent = xmalloc(sizeof(int32_t) * T);
  fork_off[0] = 0;
  ptoff[0] = 0;
  for (int t = 0; t < T; ++t) {
    fork_off[t + 1] = fork_off[t] + 1 + (int)(rnd() % 3);
    plen[t] = 1 + (int)(rnd() % 40);
    ptoff[t + 1] = ptoff[t] + (plen[t] + 15) / 16;
    parent[t] = chain ? t - 1 : -1;
  }
  const int N = fork_off[T];
  int32_t *slen = xmalloc(sizeof(int32_t) * N);
  int32_t *stoff = xmalloc(sizeof(int32_t) * (N + 1));
  stoff[0] = 0;
  for (int f = 0; f < N; ++f) {
    slen[f] = (int)(rnd() % 34);
    stoff[f + 1] = stoff[f] + (slen[f] + 15) / 16;
  }
  const int nb = ptoff[T] + stoff[N];
  int32_t *ptab = xmalloc(sizeof(int32_t) * (ptoff[T] ? ptoff[T] : 1));
  int32_t *stab = xmalloc(sizeof(int32_t) * (stoff[N] ? stoff[N] : 1));
  for (int i = 0; i < ptoff[T]; ++i) ptab[i] = nb - 1 - i;   /* reversed: ids far from their order */
  for (int i = 0; i < stoff[N]; ++i) stab[i] = nb - 1 - ptoff[T] - i;
  const int64_t elems = (int64_t)nb * Hkv * 16 * D;
  const int es = fp8 ? 1 : 2;
  uint8_t *kp = xmalloc((size_t)(elems * es));
  uint8_t *vp = xmalloc((size_t)(elems * es));
  float *ksc = fp8 ? xmalloc(sizeof(float) * nb) : NULL;
  float *vsc = fp8 ? xmalloc(sizeof(float) * nb) : NULL;
  for (int64_t i = 0; i < elems; ++i) {
    if (fp8) {
      kp[i] = (uint8_t)(rnd() % 0x77);   /* finite codes */
      vp[i] = (uint8_t)(rnd() % 0x77);
    } else {
      ((uint16_t *)kp)[i] = bf16_of(2 * unif() - 1);
      ((uint16_t *)vp)[i] = bf16_of(2 * unif() - 1);
    }
  }
  for (int i = 0; fp8 && i < nb; ++i) {
    ksc[i] = (float)(0.01 + unif());
    vsc[i] = (float)(0.01 + unif());
  }
  uint16_t *q = xmalloc(sizeof(uint16_t) * (size_t)N * Hq * D);
  for (int64_t i = 0; i < (int64_t)N * Hq * D; ++i) q[i] = bf16_of(2 * unif() - 1);
  specgen_ref_batch_t b;
  memset(&b, 0, sizeof b);
  b.num_traces = T;
  b.num_forks = N;
  b.num_q_heads = Hq;
  b.num_kv_heads = Hkv;
  b.head_dim = D;
  b.block_size = 16;
  b.num_blocks = nb;
  b.sm_scale = 1.0 / sqrt((double)D);
  b.kv_dtype = fp8;
  b.q = q;
  b.k_pool = kp;
  b.v_pool = vp;
  b.k_scale = ksc;
  b.v_scale = vsc;
  b.fork_off = fork_off;
  b.prefix_len = plen;
  b.prefix_table_off = ptoff;
  b.prefix_table = ptab;
  b.suffix_len = slen;
  b.suffix_table_off = stoff;
  b.suffix_table = stab;
  b.prefix_parent = parent;
  double *out = xmalloc(sizeof(double) * (size_t)N * Hq * D);
  double *lse = xmalloc(sizeof(double) * (size_t)N * Hq);
  if (specgen_ref_fork_decode_attn(&b, NULL, 0, out, lse, 1) != 0) FAIL("decode rejected a valid batch");
  for (int64_t i = 0; i < (int64_t)N * Hq; ++i)
    if (!isfinite(lse[i])) FAIL("non-finite lse at row %lld", (long long)i);
  /* a row subset: the last row and the first */
  int32_t rows[4] = {N - 1, Hq - 1, 0, 0};
  double out2[2 * 128], lse2[2];
  if (specgen_ref_fork_decode_attn(&b, rows, 2, out2, lse2, 1) != 0) FAIL("row subset rejected");
  if (lse2[1] != lse[0] || lse2[0] != lse[(int64_t)N * Hq - 1]) FAIL("row subset differs");
  /* prefill: forks with at least one suffix token take 1..S_f queries; the
     others are given one token of suffix first */
  int32_t *ql = xmalloc(sizeof(int32_t) * N);
  int64_t nq = 0;
  for (int f = 0; f < N; ++f) {
    ql[f] = slen[f] > 0 ? 1 + (int)(rnd() % slen[f]) : 0;
    nq += ql[f];
  }
  int ok_prefill = 1;
  for (int f = 0; f < N; ++f) ok_prefill &= ql[f] >= 1;
  if (ok_prefill) {
    uint16_t *qq = xmalloc(sizeof(uint16_t) * (size_t)nq * Hq * D);
    for (int64_t i = 0; i < nq * Hq * D; ++i) qq[i] = bf16_of(2 * unif() - 1);
    specgen_ref_batch_t bp = b;
    bp.q = qq;
    double *po = xmalloc(sizeof(double) * (size_t)nq * Hq * D);
    double *pl = xmalloc(sizeof(double) * (size_t)nq * Hq);
    if (specgen_ref_fork_prefill_attn(&bp, ql, NULL, 0, po, pl, 1) != 0) FAIL("prefill rejected");
    free(qq);
    free(po);
    free(pl);
  } else {
    if (specgen_ref_fork_prefill_attn(&b, ql, NULL, 0, out, lse, 1) != -1) FAIL("bad q_len accepted");
  }
  /* append one token per fork at its suffix length where the table has room */
  uint8_t *kn = xmalloc((size_t)N * Hkv * D * es);
  uint8_t *vn = xmalloc((size_t)N * Hkv * D * es);
  memset(kn, 0x11, (size_t)N * Hkv * D * es);
  memset(vn, 0x22, (size_t)N * Hkv * D * es);
  int32_t *pos = xmalloc(sizeof(int32_t) * N);
  for (int f = 0; f < N; ++f) pos[f] = slen[f] > 0 ? slen[f] - 1 : -1;
  int64_t skipped = specgen_ref_kv_append(kp, vp, kn, vn, es, N, Hkv, D, pos, stoff, stab, nb);
  int64_t expect = 0;
  for (int f = 0; f < N; ++f) expect += slen[f] == 0;
  if (skipped != expect) FAIL("append skipped %lld, expected %lld", (long long)skipped, (long long)expect);
  free(kn);
  free(vn);
  free(pos);
  free(ql);
  free(out);
  free(lse);
  free(q);
  free(kp);
  free(vp);
  free(ksc);
  free(vsc);
  free(ptab);
  free(stab);
  free(slen);
  free(stoff);
  free(fork_off);
  free(plen);
  free(ptoff);
  free(parent);
}

static void run_moves(void) {
  const int64_t n = 7, nb = 11, bb = 36;
  uint8_t *pool = xmalloc((size_t)(nb * bb));
  uint8_t *stg = xmalloc((size_t)(n * bb));
  int32_t ids[7] = {3, -1, 10, 0, 11, 5, 7};
  for (int64_t i = 0; i < n * bb; ++i) stg[i] = (uint8_t)rnd();
  memset(pool, 0xA5, (size_t)(nb * bb));
  if (specgen_ref_kv_import(pool, stg, bb, ids, n, nb) != 2) FAIL("import bad-id count");
  uint8_t *back = xmalloc((size_t)(n * bb));
  memset(back, 0, (size_t)(n * bb));
  if (specgen_ref_kv_export(back, pool, bb, ids, n, nb) != 2) FAIL("export bad-id count");
  for (int64_t i = 0; i < n; ++i)
    if (ids[i] >= 0 && ids[i] < nb && memcmp(back + i * bb, stg + i * bb, (size_t)bb)) FAIL("round trip");
  free(pool);
  free(stg);
  free(back);
}

static void run_merge(void) {
  const int S = 5, R = 9, D = 24;
  float *o = xmalloc(sizeof(float) * S * R * D);
  float *l = xmalloc(sizeof(float) * S * R);
  for (int i = 0; i < S * R * D; ++i) o[i] = (float)(2 * unif() - 1);
  for (int i = 0; i < S * R; ++i) l[i] = (i % 7 == 0) ? -INFINITY : (float)(10 * unif());
  for (int s = 0; s < S; ++s) l[s * R + R - 1] = -INFINITY;   /* an all-empty row */
  double *out = xmalloc(sizeof(double) * R * D);
  double *lse = xmalloc(sizeof(double) * R);
  specgen_ref_lse_merge(o, l, S, R, D, out, lse);
  if (lse[R - 1] != -INFINITY || out[(R - 1) * D] != 0.0) FAIL("empty row");
  free(o);
  free(l);
  free(out);
  free(lse);
}

static void run_decode(void) {
  uint8_t codes[256];
  uint16_t bits[256];
  double d8[256], d16[256];
  for (int i = 0; i < 256; ++i) {
    codes[i] = (uint8_t)i;
    bits[i] = (uint16_t)(i * 257);
  }
  specgen_ref_decode_e4m3(codes, 256, d8);
  specgen_ref_decode_bf16(bits, 256, d16);
  if (d8[0x38] != 1.0 || d8[0x7E] != 448.0 || !isnan(d8[0x7F])) FAIL("e4m3 decode");
  double q[3] = {1, 0, 0}, o[3], lse;
  specgen_ref_attend_dense(q, NULL, NULL, 0, 3, 1.0, o, &lse);   /* the empty set */
  if (lse != -INFINITY) FAIL("empty dense");
}

int main(int argc, char **argv) {
  const int reps = argc > 1 ? atoi(argv[1]) : 40;
  run_decode();
  run_moves();
  run_merge();
  for (int r = 0; r < reps; ++r) {
    const int T = 1 + (int)(rnd() % 4);
    const int Hkv = 1 + (int)(rnd() % 3);
    const int g = 1 + (int)(rnd() % 4);
    const int D = (rnd() & 1) ? 64 : 128;
    run_batch(T, (int)(rnd() & 1), (int)(rnd() & 1), Hkv * g, Hkv, D);
  }
  printf("OK %d batches\n", reps);
  return 0;
}
