// planner.h -- host-only construction of the work split (plan.h) from the
// host mirrors of the lengths.  Plain C++ with no HIP dependency, so it is
// also compiled by a g++ test harness that replays every worker walk and
// every merge lookup on the CPU.
#pragma once
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>

#include "plan.h"

namespace specgen {

enum { kPlanOk = 0, kPlanInvalid = 1, kPlanUnsupported = 2 };

struct PlanInputs {
  int T, N, Hq, Hkv, D, policy;
  const int32_t* fork_off;    // [T+1]
  const int32_t* prefix_parent;  // [T] parent trace or -1, or NULL (every trace a root)
  const int32_t* prefix_in_suffix_table;  // [T] 1: trace t's prefix ids index the suffix table; or NULL
  const int32_t* prefix_len;  // [T]
  const int32_t* suffix_len;  // [N]
  const int32_t* prefix_table_off;  // [T+1]
  const int32_t* suffix_table_off;  // [N+1]
  int tt[2];                  // tokens per tile, per partition
  int rbs[2];                 // rows per row block
  int item_cap[2];            // max items per worker
  int tile_cap[2];            // max tiles per worker
  int walk_threads[2];        // threads of a parallel walk (0: serial walk, no unit limit)
  int charge[2];              // units in front of every prefix item
  int charge_suf[2];          // units in front of every suffix item
  int wt_rg[2][9];            // units per tile of an item of 1..8 row groups of 32 rows ([0] unused)
};

// Row groups of 32 rows of an item of `rows` rows (at most 8: row blocks hold
// at most 256 rows).
inline int row_groups(int rows) { return rows <= 32 ? 1 : rows >= 225 ? 8 : (rows + 31) / 32; }

constexpr int64_t kAlignFloats = 64;   // 256-byte alignment of workspace regions

inline int64_t align_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

// Validates shapes and lengths, fills `plan` and the workspace size in floats.
// `cus` returns the number of compute units (workers per partition start at it).
template <typename CusFn>
int plan_build(const PlanInputs& in, CusFn cus_fn, Plan* plan, int64_t* ws_floats, char* err, size_t errlen) {
#define SG_FAIL(code, ...)                 \
  do {                                     \
    snprintf(err, errlen, __VA_ARGS__);    \
    return code;                           \
  } while (0)
  const int T = in.T, N = in.N, Hq = in.Hq, Hkv = in.Hkv, D = in.D;
  if (T < 1) SG_FAIL(kPlanInvalid, "num_traces must be >= 1 (got %d)", T);
  if (N < 1) SG_FAIL(kPlanInvalid, "num_forks must be >= 1 (got %d)", N);
  if (T > kMaxTraces) SG_FAIL(kPlanUnsupported, "num_traces %d exceeds %d per call", T, kMaxTraces);
  if (N > kMaxForks) SG_FAIL(kPlanUnsupported, "num_forks %d exceeds %d per call", N, kMaxForks);
  if (Hq < 1 || Hkv < 1 || Hq % Hkv != 0)
    SG_FAIL(kPlanInvalid, "num_q_heads %d must be a positive multiple of num_kv_heads %d", Hq, Hkv);
  if (Hq / Hkv > 128) SG_FAIL(kPlanUnsupported, "GQA group size %d exceeds 128", Hq / Hkv);
  if (D != 64 && D != 128) SG_FAIL(kPlanUnsupported, "head_dim %d not in {64, 128}", D);
  const int32_t* fo = in.fork_off;
  if (fo[0] != 0 || fo[T] != N) SG_FAIL(kPlanInvalid, "fork_off must start at 0 and end at num_forks");
  for (int t = 0; t < T; ++t) {
    if (fo[t + 1] < fo[t]) SG_FAIL(kPlanInvalid, "fork_off must be nondecreasing (trace %d)", t);
    if (in.prefix_len[t] < 1) SG_FAIL(kPlanInvalid, "prefix_len[%d] must be >= 1", t);
  }
  for (int f = 0; f < N; ++f)
    if (in.suffix_len[f] < 0) SG_FAIL(kPlanInvalid, "suffix_len[%d] must be >= 0", f);
  // Nested prefixes: each parent comes earlier, and the traces are in
  // depth-first order (a trace's parent is the previous trace or one of its
  // ancestors), so every subtree is a contiguous run of traces and forks.
  int32_t parent[kMaxTraces], depth[kMaxTraces], sub_end[kMaxTraces];
  int max_depth = 1;
  for (int t = 0; t < T; ++t) {
    const int pa = in.prefix_parent ? in.prefix_parent[t] : -1;
    if (pa < -1 || pa >= t) SG_FAIL(kPlanInvalid, "prefix_parent[%d] = %d must be -1 or an earlier trace", t, pa);
    if (pa >= 0) {
      int a = t - 1;
      while (a >= 0 && a != pa) a = parent[a];
      if (a != pa) SG_FAIL(kPlanInvalid, "traces are not in depth-first order at trace %d", t);
    }
    parent[t] = pa;
    depth[t] = pa < 0 ? 1 : depth[pa] + 1;
    if (depth[t] > kMaxDepth) SG_FAIL(kPlanUnsupported, "prefix chain deeper than %d traces", kMaxDepth);
    max_depth = std::max(max_depth, depth[t]);
  }
  for (int t = T - 1; t >= 0; --t) {   // one past the last trace of t's subtree
    sub_end[t] = t + 1;
    while (sub_end[t] < T && depth[sub_end[t]] > depth[t]) sub_end[t] = sub_end[sub_end[t]];
    // a trace may have no forks of its own only if traces nested below it have some
    if (fo[sub_end[t]] <= fo[t]) SG_FAIL(kPlanInvalid, "trace %d has no forks", t);
  }

  const int g = Hq / Hkv;
  memset(plan, 0, sizeof(Plan));
  plan->T = T;
  plan->N = N;
  plan->Hq = Hq;
  plan->Hkv = Hkv;
  plan->g = g;
  plan->D = D;
  plan->policy = in.policy;
  plan->depth = max_depth;
  for (int t = 0; t <= T; ++t) plan->fork_off[t] = fo[t];
  for (int t = 0; t < T; ++t) {
    plan->parent[t] = parent[t];
    plan->fork_end[t] = fo[sub_end[t]];
    plan->ptab_sel[t] = in.prefix_in_suffix_table ? (in.prefix_in_suffix_table[t] != 0) : 0;
  }
  for (int t = 0; t < T; ++t) plan->prefix_len[t] = in.prefix_len[t];
  for (int t = 0; t <= T; ++t) plan->prefix_table_off[t] = in.prefix_table_off[t];
  for (int f = 0; f < N; ++f) plan->suffix_len[f] = in.suffix_len[f];
  for (int f = 0; f <= N; ++f) plan->suffix_table_off[f] = in.suffix_table_off[f];
  const int xs = part_of_suffix(in.policy);
  int64_t unit_cap[2];   // units per worker a kernel's walk can take

  // prefix items, traces grouped by partition
  int pos = 0;
  for (int X = 0; X < 2; ++X) {
    PartPlan& pp = plan->part[X];
    pp.tt = in.tt[X];
    pp.rbs = in.rbs[X];
    pp.slot_rows = in.rbs[X];
    pp.trace_begin = pos;
    pp.charge = in.charge[X];
    pp.charge_suf = in.charge_suf[X];
    for (int r = 1; r <= 8; ++r)
      if (in.wt_rg[X][r] < 1) SG_FAIL(kPlanInvalid, "unit prices must be positive");
    if (pp.charge < 0 || pp.charge_suf < 0) SG_FAIL(kPlanInvalid, "unit prices must be positive");
    pp.wt_suf = in.wt_rg[X][row_groups(std::min(g, pp.rbs))];
    pp.wt_max = pp.wt_suf;
    int wt_min = pp.wt_suf;
    int64_t units = 0, items = 0;
    for (int t = 0; t < T; ++t) {
      const int rows = (plan->fork_end[t] - fo[t]) * g;   // the forks of t and its descendants
      if (part_of_trace(in.policy, rows) != X) continue;
      plan->trace_part[t] = X;
      plan->trace_pos[t] = pos;
      plan->ptrace[pos] = t;
      plan->unitP[pos] = (int32_t)units;
      plan->ordP[pos] = (int32_t)items;
      // one price for all the trace's prefix items: that of its first (fullest) row block
      plan->wtP[pos] = in.wt_rg[X][row_groups(std::min(rows, pp.rbs))];
      pp.wt_max = std::max(pp.wt_max, plan->wtP[pos]);
      wt_min = std::min(wt_min, plan->wtP[pos]);
      const int rb = cdiv(rows, pp.rbs);
      units += (int64_t)Hkv * rb * ((int64_t)cdiv(in.prefix_len[t], pp.tt) * plan->wtP[pos] + pp.charge);
      items += (int64_t)Hkv * rb;
      if (units > INT32_MAX || items > INT32_MAX) SG_FAIL(kPlanUnsupported, "batch too large");
      ++pos;
    }
    pp.n_traces = pos - pp.trace_begin;
    // a parallel walk examines chunks of at most min(price, charges) units per
    // thread, so that a chunk holds at most one tile start
    unit_cap[X] = in.walk_threads[X] > 0
                      ? (int64_t)in.walk_threads[X] * std::max(1, std::min(wt_min, std::min(pp.charge, pp.charge_suf)))
                      : INT64_MAX;
    pp.prefix_units = units;
    pp.n_prefix_items = (int32_t)items;
    pp.units = units;
    pp.has_suffix = (X == xs);
    pp.suffix_rb = cdiv(g, pp.rbs);
  }
  // suffix items, all in one partition
  {
    PartPlan& pp = plan->part[xs];
    int64_t acc = 0;
    for (int f = 0; f < N; ++f) {
      plan->unitS[f] = (int32_t)acc;
      if (in.suffix_len[f] > 0)
        acc += (int64_t)Hkv * pp.suffix_rb * ((int64_t)cdiv(in.suffix_len[f], pp.tt) * pp.wt_suf + pp.charge_suf);
      if (acc > INT32_MAX) SG_FAIL(kPlanUnsupported, "batch too large");
    }
    plan->unitS[N] = (int32_t)acc;
    pp.units += acc;
    if (pp.units > INT32_MAX) SG_FAIL(kPlanUnsupported, "batch too large");
    if ((int64_t)pp.n_prefix_items + (int64_t)N * Hkv * pp.suffix_rb > INT32_MAX)
      SG_FAIL(kPlanUnsupported, "batch too large");
  }
  // workers: one per compute unit, more while a worker's range would exceed
  // the kernel's per-worker capacity (items it can describe, units it walks,
  // tiles it can hold)
  int64_t off = 0;
  for (int X = 0; X < 2; ++X) {
    PartPlan& pp = plan->part[X];
    pp.workers = 0;
    pp.kmax = 0;
    if (pp.units == 0) continue;
    // Every worker's range spans at least the largest tile price, so each
    // worker between the first and the last of an item's workers holds a tile
    // of it (the merge takes one part from each of them).
    const int64_t wcap = std::max<int64_t>(1, pp.units / pp.wt_max);
    int64_t W = std::min<int64_t>(wcap, (int64_t)cus_fn());
    int tmax = 0;   // most tiles any worker holds
    for (;;) {
      pp.workers = (int32_t)W;
      pp.per_lo = (int32_t)(pp.units / W);
      pp.n_hi = (int32_t)(pp.units % W);
      const int64_t per = (pp.units + W - 1) / W;
      int kmax = 0;
      tmax = 0;
      for (int64_t w = 0; w < W; ++w) {
        const int64_t a = worker_start(pp, w), e = worker_start(pp, w + 1);
        if (e <= a) continue;
        const int k = locate(*plan, X, e - 1).ord - locate(*plan, X, a).ord + 1;
        if (k > kmax) kmax = k;
        const int tiles = walk_range(*plan, X, w, INT32_MAX, [](const ItemRef&, int, int, int, int) {}).R;
        if (tiles > tmax) tmax = tiles;
      }
      pp.kmax = kmax;
      if ((per <= unit_cap[X] && tmax <= in.tile_cap[X] && kmax <= in.item_cap[X]) || W == wcap) break;
      W = std::min<int64_t>(wcap, W * 2);
    }
    if (pp.kmax > in.item_cap[X] || tmax > in.tile_cap[X] || (pp.units + pp.workers - 1) / pp.workers > unit_cap[X])
      SG_FAIL(kPlanUnsupported, "work split exceeds the kernel's per-worker capacity");
    // Rows per slot: the partition's largest item, rounded up to 16 rows (an
    // MFMA N-tile stores all its 16 rows), at most the row-block size.
    int max_rows = pp.has_suffix ? std::min(g, pp.rbs) : 1;
    for (int i = pp.trace_begin; i < pp.trace_begin + pp.n_traces; ++i)
      max_rows = std::max(max_rows, std::min(trace_rows(*plan, plan->ptrace[i]), pp.rbs));
    pp.slot_rows = std::min(pp.rbs, (max_rows + 15) / 16 * 16);
    const int64_t slots = (int64_t)pp.workers * pp.kmax;
    // o: fp16 [slots][slot_rows][D] (D is even); lse: (lse, dec) float pairs
    pp.o_base = off;
    off = align_up(off + slots * pp.slot_rows * D / 2, kAlignFloats);
    pp.lse_base = off;
    off = align_up(off + 2 * slots * pp.slot_rows, kAlignFloats);
    pp.n_items = pp.n_prefix_items + (pp.has_suffix ? N * Hkv * pp.suffix_rb : 0);
    pp.info_base = off;
    off = align_up(off + 3 * (int64_t)pp.n_items, kAlignFloats);
  }
  *ws_floats = off;
  return kPlanOk;
#undef SG_FAIL
}

}  // namespace specgen
