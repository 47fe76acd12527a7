// plan.h -- the work split of fork-decode attention, shared by the host
// planner and the kernels (all functions are __host__ __device__).
//
// Work items.  A prefix item is (trace t, kv head j, row block rb): the rows
// are every (fork of t, q head of j's group) pair, F_t * g of them, cut into
// blocks of `rbs` rows; it streams the trace's P_t prefix tokens of head j
// once for all those rows, which is the point of forking off a shared prefix
// (the forks reuse the reasoning prefix's KV, Sec. 4.2 and Sec. 8.7).  A
// suffix item is (fork f, kv head j, row block rb) over the fork's own S_f
// tokens with the g query heads of the group as rows.
//
// Partitions.  Each item is served by one of two kernels (0 = MFMA, 1 = dot),
// chosen by the path policy.  Within a partition the items are laid out in a
// fixed order -- prefix items (trace-major, then j, then rb), then suffix
// items (fork-major, then j, then rb) -- and each item is cut into tiles of
// `tt` tokens.
//
// Units.  The split is made over a sequence of units that prices the work:
// every item first takes units for its fixed cost in a worker (its query rows
// and its end: `charge` for a prefix item, `charge_suf` for a suffix item),
// then a price per tile that grows with the rows the item computes: wtP[] for
// the prefix items of each trace, wt_suf for suffix items (g rows of one
// fork).  The sequence is split evenly over W
// workers (workgroups): worker w takes units [start(w), start(w+1)) and
// processes the tiles whose first unit lies there.  A worker emits one partial
// (o, lse) per item it touches, into slot w * kmax + k where k is the item's
// ordinal minus the ordinal of the item at the worker's first unit.  The merge
// finds the workers covering an item from its units alone.
#pragma once
#include <stdint.h>

#ifdef __HIPCC__
#define SG_HD __host__ __device__ __forceinline__
#else
#define SG_HD inline
#endif

namespace specgen {

constexpr int kMaxTraces = 32;   // traces per call
constexpr int kMaxForks = 512;   // forks per call
constexpr int kMaxDepth = 8;     // traces on one prefix chain (nested prefixes)
constexpr int kBlock = 16;       // tokens per KV block

enum { kPartMfma = 0, kPartDot = 1 };
enum { kPolicyAuto = 0, kPolicyDot = 1, kPolicyMfma = 2 };

struct PartPlan {
  int64_t units;          // total units of the partition
  int64_t prefix_units;   // units of its prefix items (they come first)
  int64_t o_base;         // float offset of slot 0's o (fp16 rows, see part_row_k) in the workspace
  int64_t lse_base;       // float offset of slot 0's (lse, dec) pairs
  int64_t info_base;      // float offset of the item table: per item ordinal three
                          // int32 (first worker, last worker, segment index in the first)
  int32_t n_items;        // items of the partition (prefix, then suffix)
  int32_t per_lo;         // units / W: every worker gets per_lo units, the first
  int32_t n_hi;           // units % W workers one more
  int32_t workers;        // W (0: partition unused)
  int32_t kmax;           // max items touched by one worker
  int32_t tt;             // tokens per tile
  int32_t rbs;            // rows per row block
  int32_t slot_rows;      // rows reserved per partial slot: the largest item's, rounded up to 16
  int32_t n_prefix_items; // prefix items in the partition
  int32_t has_suffix;     // suffix items belong to this partition
  int32_t suffix_rb;      // row blocks per suffix (fork, head): ceil(g / rbs)
  int32_t n_traces;       // traces whose prefix items are in the partition
  int32_t trace_begin;    // their positions in Plan::ptrace: [trace_begin, +n_traces)
  int32_t charge;         // units in front of every prefix item (its fixed cost)
  int32_t charge_suf;     // units in front of every suffix item
  int32_t wt_suf;         // units per tile of a suffix item
  int32_t wt_max;         // the largest tile price of the partition
};

// The scalar part of the plan.
struct PlanHead {
  int32_t T, N, Hq, Hkv, g, D;
  int32_t policy;
  int32_t depth;          // traces on the longest prefix chain (1: no nesting)
  PartPlan part[2];
};

// The whole plan, computed on the host from the length mirrors and passed to
// every kernel by value (about 7.8 KB of kernel arguments); each workgroup
// copies it into LDS with one vector load per thread (plan_to_lds).
struct alignas(16) Plan : PlanHead {
  int32_t fork_off[kMaxTraces + 1];
  int32_t prefix_len[kMaxTraces];
  // Nested prefixes: a fork of trace t attends over the prefix tokens of
  // every trace on the chain root, ..., parent[t], t.  Traces are in
  // depth-first order, so the forks of t and its descendants are
  // [fork_off[t], fork_end[t]): the rows of t's prefix items.
  int32_t parent[kMaxTraces];       // -1 for a root
  int32_t fork_end[kMaxTraces];
  // 1: trace t's prefix blocks are listed in the suffix table (a prefill
  // shares the whole blocks before a fork's first query as a nested prefix)
  int32_t ptab_sel[kMaxTraces];
  int32_t trace_part[kMaxTraces];   // partition of trace t's prefix items
  int32_t trace_pos[kMaxTraces];    // index of t in ptrace
  int32_t ptrace[kMaxTraces];       // traces grouped by partition, ascending within each
  int32_t unitP[kMaxTraces];        // (by ptrace position) first unit of the trace's prefix items
  int32_t ordP[kMaxTraces];         // (by ptrace position) ordinal of its first prefix item
  int32_t wtP[kMaxTraces];          // (by ptrace position) units per tile of its prefix items
  int32_t unitS[kMaxForks + 1];     // first unit of fork f's suffix items, relative to prefix_units
  int32_t prefix_table_off[kMaxTraces + 1];   // host mirrors of the batch's index arrays
  int32_t suffix_len[kMaxForks];
  int32_t suffix_table_off[kMaxForks + 1];
};

SG_HD int32_t cdiv(int64_t a, int64_t b) { return (int32_t)((a + b - 1) / b); }
SG_HD int32_t cdiv32(int32_t a, int32_t b) { return (a + b - 1) / b; }



SG_HD int32_t trace_rows(const Plan& p, int t) { return (p.fork_end[t] - p.fork_off[t]) * p.g; }

SG_HD int part_of_trace(int policy, int rows) {
  if (policy == kPolicyDot) return kPartDot;
  if (policy == kPolicyMfma) return kPartMfma;
  return rows >= 16 ? kPartMfma : kPartDot;
}

SG_HD int part_of_suffix(int policy) { return policy == kPolicyDot ? kPartDot : kPartMfma; }

// First unit of worker w: workers [0, n_hi) take per_lo + 1 units, the rest
// per_lo (no division, so the kernels evaluate it cheaply).
SG_HD int64_t worker_start(const PartPlan& pp, int64_t w) {
  return w * pp.per_lo + (w < pp.n_hi ? w : (int64_t)pp.n_hi);
}

#ifdef __HIPCC__
// Copy the plan from the kernel arguments into LDS.  All kThreads threads of
// the block call this; it ends with a barrier.
template <int kThreads>
__device__ __forceinline__ void plan_to_lds(const Plan& karg, Plan& p) {
  static_assert(sizeof(Plan) % 16 == 0, "plan copies in 16-byte pieces");
  constexpr int kPieces = (int)(sizeof(Plan) / 16);
  typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
  const u32x4_t* src = reinterpret_cast<const u32x4_t*>(&karg);
  u32x4_t* dst = reinterpret_cast<u32x4_t*>(&p);
  for (int i = threadIdx.x; i < kPieces; i += kThreads) dst[i] = src[i];
  __syncthreads();
}
#endif

// Worker owning unit x: the largest w with worker_start(w) <= x.  Units fit
// in 32 bits (the planner rejects larger partitions), so the divisions are
// 32-bit.
SG_HD int32_t worker_of_unit(const PartPlan& pp, int64_t x) {
  const uint32_t big = (uint32_t)pp.n_hi * (uint32_t)(pp.per_lo + 1);   // units of the larger ranges
  const uint32_t xx = (uint32_t)x;
  if (xx < big) return (int32_t)(xx / (uint32_t)(pp.per_lo + 1));
  return (int32_t)((uint32_t)pp.n_hi + (xx - big) / (uint32_t)pp.per_lo);
}

struct ItemRef {
  int32_t kind;      // 0 prefix, 1 suffix, -1 past the end
  int32_t t, f, j, rb;
  int32_t tiles;     // tiles of the item (its data)
  int32_t w;         // units per tile of the item
  int32_t off;       // units from the start of the item's tile 0 to x (< 0 in its charge)
  int32_t tile;      // tile holding x (off / w), -1 in the charge
  int64_t first;     // sequence unit where the item's tile 0 starts
  int32_t ord;       // ordinal of the item in the partition
};

// Units taken by one suffix item of fork f (0 if S_f = 0): charge_suf plus
// ceil(S_f / tt) tiles of wt_suf units; unitS holds their per-fork prefix sums.
SG_HD int32_t suffix_span(const Plan& p, const PartPlan& pp, int f) {
  return (p.unitS[f + 1] - p.unitS[f]) / (p.Hkv * pp.suffix_rb);
}

// The item at partition sequence unit x.
SG_HD ItemRef locate(const Plan& p, int part, int64_t x) {
  const PartPlan& pp = p.part[part];
  ItemRef r;
  r.kind = -1;
  r.t = r.f = r.j = r.rb = r.tiles = r.tile = r.off = r.ord = 0;
  r.w = 1;
  r.first = 0;
  if (x < 0 || x >= pp.units) return r;
  int local, span, item, charge;
  if (x < pp.prefix_units) {
    // largest position i in the partition's trace list with unitP[i] <= x
    int lo = pp.trace_begin, hi = pp.trace_begin + pp.n_traces - 1;
    while (lo < hi) {
      int mid = (lo + hi + 1) >> 1;
      if (p.unitP[mid] <= x) lo = mid; else hi = mid - 1;
    }
    const int t = p.ptrace[lo];
    const int rb_count = cdiv32(trace_rows(p, t), pp.rbs);
    r.tiles = cdiv32(p.prefix_len[t], pp.tt);
    r.w = p.wtP[lo];
    charge = pp.charge;
    span = r.tiles * r.w + charge;
    local = (int)(x - p.unitP[lo]);   // unit counts fit in int32 (the planner checks)
    item = local / span;
    r.kind = 0;
    r.t = t;
    r.j = item / rb_count;
    r.rb = item % rb_count;
    r.ord = p.ordP[lo] + item;
  } else {
    const int xs = (int)(x - pp.prefix_units);
    int lo = 0, hi = p.N - 1;   // largest f with unitS[f] <= xs
    while (lo < hi) {
      int mid = (lo + hi + 1) >> 1;
      if (p.unitS[mid] <= xs) lo = mid; else hi = mid - 1;
    }
    const int f = lo;
    span = suffix_span(p, pp, f);
    r.w = pp.wt_suf;
    charge = pp.charge_suf;
    r.tiles = (span - charge) / r.w;
    local = xs - p.unitS[f];
    item = local / span;
    r.kind = 1;
    r.f = f;
    r.j = item / pp.suffix_rb;
    r.rb = item % pp.suffix_rb;
    r.ord = pp.n_prefix_items + (f * p.Hkv + r.j) * pp.suffix_rb + r.rb;
  }
  r.off = local - item * span - charge;
  r.tile = r.off >= 0 ? r.off / r.w : -1;
  r.first = x - r.off;
  return r;
}

// The item that follows `cur` in partition `part` (cur must not be the last
// one), with x at its tile 0: equal to locate(p, part, x) for x = cur.first +
// cur.tiles * cur.w + the next item's charge.  Steps within a trace or fork
// in O(1) and falls back to locate() where it would have to skip over forks
// without suffix tokens or cross into the suffix items.
SG_HD ItemRef next_item(const Plan& p, int part, const ItemRef& cur) {
  const PartPlan& pp = p.part[part];
  const int64_t end = cur.first + (int64_t)cur.tiles * cur.w;   // where the next item's charge starts
  ItemRef r = cur;
  r.first = end + (cur.kind == 0 ? pp.charge : pp.charge_suf);
  r.tile = 0;
  r.off = 0;
  r.ord = cur.ord + 1;
  if (cur.kind == 0) {
    const int rb_count = cdiv32(trace_rows(p, cur.t), pp.rbs);
    if (cur.rb + 1 < rb_count) {
      r.rb = cur.rb + 1;
      return r;
    }
    if (cur.j + 1 < p.Hkv) {
      r.j = cur.j + 1;
      r.rb = 0;
      return r;
    }
    const int pos = p.trace_pos[cur.t] + 1;
    if (pos < pp.trace_begin + pp.n_traces) {
      r.t = p.ptrace[pos];
      r.j = 0;
      r.rb = 0;
      r.tiles = cdiv32(p.prefix_len[r.t], pp.tt);
      r.w = p.wtP[pos];
      return r;
    }
  } else if (cur.rb + 1 < pp.suffix_rb) {
    r.rb = cur.rb + 1;
    return r;
  } else if (cur.j + 1 < p.Hkv) {
    r.j = cur.j + 1;
    r.rb = 0;
    return r;
  } else if (cur.f + 1 < p.N) {
    const int f = cur.f + 1;
    const int span = suffix_span(p, pp, f);
    if (span > 0) {
      r.f = f;
      r.j = 0;
      r.rb = 0;
      r.tiles = (span - pp.charge_suf) / pp.wt_suf;
      return r;
    }
  }
  r = locate(p, part, end);   // at the first unit of the next item's charge
  r.tile = 0;
  r.off = 0;
  return r;
}

// The items of worker w's range, in order.  For each one with tiles in the
// range (tiles whose first unit lies in it) calls visit(it, n, rt, i, k): it =
// the item (it.tile = its first tile in the range), n = its tiles in the
// range, rt = the number of tiles of the range before them, i = its position
// among the visited items, k = it.ord - (ordinal of the item at the range's
// first unit), which is the partial-slot index (w * kmax + k).  At most
// item_cap items are visited.
struct WorkerRange {
  int nitems;     // items visited
  int first_ord;  // ordinal of the item at the range's first unit
  int R;          // tiles in the range
};
template <typename Visit>
SG_HD WorkerRange walk_range(const Plan& p, int part, int64_t w, int item_cap, Visit&& visit) {
  const PartPlan& pp = p.part[part];
  const int64_t x0 = worker_start(pp, w);
  const int64_t x1 = worker_start(pp, w + 1);
  WorkerRange wr;
  wr.nitems = 0;
  wr.first_ord = 0;
  wr.R = 0;
  if (x0 >= x1) return wr;
  ItemRef it = locate(p, part, x0);
  wr.first_ord = it.ord;
  int t = it.off <= 0 ? 0 : cdiv32(it.off, it.w);   // first tile starting at or after x0
  for (;;) {
    const int64_t u = it.first + (int64_t)t * it.w;   // where tile t starts
    if (u >= x1) break;
    if (t < it.tiles) {
      if (wr.nitems >= item_cap) break;
      const int left = cdiv(x1 - u, it.w);            // tile starts left in the range
      const int n = (it.tiles - t) < left ? (it.tiles - t) : left;
      ItemRef v = it;
      v.tile = t;
      v.off = t * it.w;
      visit(v, n, wr.R, wr.nitems, it.ord - wr.first_ord);
      wr.R += n;
      ++wr.nitems;
      if (t + n < it.tiles) break;   // the range ends inside this item
    }
    const int64_t end = it.first + (int64_t)it.tiles * it.w;   // where the next item's charge starts
    if (end >= pp.units || end + (end >= pp.prefix_units ? pp.charge_suf : pp.charge) >= x1) break;
    it = next_item(p, part, it);
    t = 0;
  }
  return wr;
}

// The parallel form of walk_range: what the chunk [u0, u0 + c) of worker w's
// range [x0, x1) contributes, for chunks no longer than any tile price or the
// charge (so a chunk holds at most one tile start, and the next item's tile 0
// never shares a chunk with the tile start it follows).  `data` marks a tile
// starting in the chunk (it.tile = that tile); `starts` marks the first tile
// of an item's segment in the range (the item's tile 0, or its first tile at
// or after x0); there, n is the segment's length in tiles.  The segments in
// order of u0 are exactly walk_range's visits: the visit index of a segment is
// the number of starting chunks before it, its rt the number of data chunks
// before it, and its slot index it.ord minus the ordinal of the item at x0.
struct TileInRange {
  ItemRef it;
  bool data;
  bool starts;
  int n;
};
SG_HD TileInRange tile_in_chunk(const Plan& p, int part, int64_t x0, int64_t x1, int64_t u0, int c) {
  TileInRange r;
  r.it = locate(p, part, u0);
  r.data = r.starts = false;
  r.n = 0;
  if (r.it.kind < 0) return r;
  const int w = r.it.w;
  const int t = r.it.off <= 0 ? 0 : cdiv32(r.it.off, w);   // first tile starting at or after u0
  if (t >= r.it.tiles) return r;
  const int64_t s = r.it.first + (int64_t)t * w;
  if (s >= u0 + c || s >= x1) return r;
  r.it.tile = t;
  r.it.off = t * w;
  r.data = true;
  r.starts = t == 0 || s - w < x0;
  const int left = cdiv(x1 - s, w);
  r.n = (r.it.tiles - t) < left ? (r.it.tiles - t) : left;
  return r;
}

// The item-table entry a walk records: the worker holding an item's first
// tile stores itself and the item's slot index there, the worker holding its
// last tile stores itself.  info holds three int32 per item ordinal.
SG_HD void record_item(int32_t* info, const ItemRef& it, int n, int w, int k) {
  if (it.tile == 0) {
    info[3 * it.ord + 0] = w;
    info[3 * it.ord + 2] = k;
  }
  if (it.tile + n == it.tiles) info[3 * it.ord + 1] = w;
}

// Trace of fork f (fork_off is nondecreasing; empty traces are rejected).
SG_HD int trace_of_fork(const Plan& p, int f) {
  int lo = 0, hi = p.T - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (p.fork_off[mid] <= f) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// (fork, q head) of row rr of an item whose first row is row0.
SG_HD void item_row_fork_head(const Plan& p, int kind, int t, int f, int j, int row0, int rr, int* fork, int* head) {
  if (kind == 0) {
    const int ri = row0 + rr;
    *fork = p.fork_off[t] + ri / p.g;
    *head = j * p.g + ri % p.g;
  } else {
    *fork = f;
    *head = j * p.g + row0 + rr;
  }
}

// The partial results of one item: workers w_lo..w_hi of partition `part`
// covered its tiles; in w_lo it is segment k_lo, in every later one segment 0
// (their ranges start inside the item).
struct ItemParts {
  int part;
  int w_lo, w_hi;
  int k_lo;
  int row;         // row inside the item
};

SG_HD ItemParts item_parts(const Plan& p, int part, int64_t first_unit, int tiles, int w, int ord, int row) {
  const PartPlan& pp = p.part[part];
  ItemParts ip;
  ip.part = part;
  ip.row = row;
  ip.w_lo = worker_of_unit(pp, first_unit);
  ip.w_hi = worker_of_unit(pp, first_unit + (int64_t)(tiles - 1) * w);
  const ItemRef f0 = locate(p, part, worker_start(pp, ip.w_lo));
  ip.k_lo = ord - f0.ord;
  return ip;
}

// The prefix item of trace t (the fork's own trace or one of its ancestors)
// that holds row (f, h), and the row inside the item.
SG_HD ItemParts prefix_parts_of_row(const Plan& p, int f, int h, int t) {
  const int g = p.g, j = h / g, hh = h - j * g;
  const int ri = (f - p.fork_off[t]) * g + hh;
  const int X = p.trace_part[t];
  const PartPlan& pp = p.part[X];
  const int rbc = cdiv32(trace_rows(p, t), pp.rbs);
  const int rb = ri / pp.rbs;
  const int tiles = cdiv32(p.prefix_len[t], pp.tt);
  const int pos = p.trace_pos[t];
  const int item = j * rbc + rb;
  return item_parts(p, X, (int64_t)p.unitP[pos] + (int64_t)item * (tiles * p.wtP[pos] + pp.charge) + pp.charge, tiles,
                    p.wtP[pos], p.ordP[pos] + item, ri - rb * pp.rbs);
}

// The suffix item of row (f, h); returns false if the fork has no suffix tokens.
SG_HD bool suffix_parts_of_row(const Plan& p, int f, int h, ItemParts* out) {
  const int g = p.g, j = h / g, hh = h - j * g;
  const int X = part_of_suffix(p.policy);
  const PartPlan& pp = p.part[X];
  const int per_fork = p.Hkv * pp.suffix_rb;
  const int span = suffix_span(p, pp, f);
  if (span <= 0) return false;
  const int rb = hh / pp.rbs;
  const int item = j * pp.suffix_rb + rb;
  *out = item_parts(p, X, pp.prefix_units + p.unitS[f] + (int64_t)item * span + pp.charge_suf,
                    (span - pp.charge_suf) / pp.wt_suf, pp.wt_suf, pp.n_prefix_items + f * per_fork + item,
                    hh - rb * pp.rbs);
  return true;
}

// The prefix item of trace t that holds row (f, h): its partition, ordinal
// and the row inside it (t is the fork's own trace or one of its ancestors).
SG_HD void prefix_item_of_row(const Plan& p, int f, int h, int t, int* part, int* ord, int* row) {
  const int g = p.g, j = h / g, hh = h - j * g;
  const int ri = (f - p.fork_off[t]) * g + hh;
  const int X = p.trace_part[t];
  const PartPlan& pp = p.part[X];
  const int rbc = cdiv32(trace_rows(p, t), pp.rbs);
  const int rb = ri / pp.rbs;
  *part = X;
  *ord = p.ordP[p.trace_pos[t]] + j * rbc + rb;
  *row = ri - rb * pp.rbs;
}

// The suffix item of row (f, h); false if the fork has no suffix tokens.
SG_HD bool suffix_item_of_row(const Plan& p, int f, int h, int* part, int* ord, int* row) {
  const int g = p.g, j = h / g, hh = h - j * g;
  const int X = part_of_suffix(p.policy);
  const PartPlan& pp = p.part[X];
  if (p.unitS[f + 1] == p.unitS[f]) return false;
  const int rb = hh / pp.rbs;
  *part = X;
  *ord = pp.n_prefix_items + (f * p.Hkv + j) * pp.suffix_rb + rb;
  *row = hh - rb * pp.rbs;
  return true;
}

// The most partial results any output row merges (host): over the chain of
// prefix items a row can see (at most `depth`) and its suffix item, the
// workers each item's tiles span.
inline int max_parts_per_row(const Plan& p) {
  int mp = 0, ms = 0;
  for (int t = 0; t < p.T; ++t) {
    const PartPlan& pp = p.part[p.trace_part[t]];
    const int rows = trace_rows(p, t);
    for (int j = 0; j < p.Hkv; ++j)
      for (int r0 = 0; r0 < rows; r0 += pp.rbs) {   // one row of each row block
        const ItemParts P = prefix_parts_of_row(p, p.fork_off[t] + r0 / p.g, j * p.g + r0 % p.g, t);
        mp = mp > P.w_hi - P.w_lo + 1 ? mp : P.w_hi - P.w_lo + 1;
      }
  }
  const PartPlan& ps = p.part[part_of_suffix(p.policy)];
  for (int f = 0; f < p.N; ++f)
    for (int j = 0; j < p.Hkv; ++j)
      for (int hh = 0; hh < p.g; hh += ps.rbs) {
        ItemParts S;
        if (suffix_parts_of_row(p, f, j * p.g + hh, &S)) ms = ms > S.w_hi - S.w_lo + 1 ? ms : S.w_hi - S.w_lo + 1;
      }
  return p.depth * mp + ms;
}

// Storage of one partial row.  The normalised partial output o (a convex
// combination of value rows) is kept as fp16 times a power of two chosen per
// row: with mx = max_d |o_d| and e its biased fp32 exponent, k = clamp(e - 14,
// 1, 240), the row stores fp16(o_d * 2^(127-k)) (so its largest element lies
// in [2^14, 2^15)) and, beside its lse, dec = 2^(k-127), so o_d = stored_d *
// dec.  Any finite o fits, and each element keeps fp16's 11-bit significand
// relative to the row's largest: the rounding is 2^-12 of mx at most, 8x
// below the bf16 rounding of the final output.
SG_HD int32_t part_row_k(uint32_t mx_bits) {
  const int32_t e = (int32_t)((mx_bits >> 23) & 0xFF);
  const int32_t k = e - 14;
  return k < 1 ? 1 : (k > 240 ? 240 : k);
}
// float offsets of the o row (fp16: 2 per float) and of the (lse, dec) pair
SG_HD int64_t part_o_off(const PartPlan& pp, int64_t slot, int row, int D) {
  return pp.o_base + (slot * pp.slot_rows + row) * (int64_t)(D / 2);
}
SG_HD int64_t part_l_off(const PartPlan& pp, int64_t slot, int row) {
  return pp.lse_base + 2 * (slot * pp.slot_rows + row);
}

// Partial-slot index of (worker w, item of ordinal ord), or -1 if out of range.
SG_HD int64_t slot_of(const PartPlan& pp, int32_t w, int32_t k) {
  if (k < 0 || k >= pp.kmax || w < 0 || w >= pp.workers) return -1;
  return (int64_t)w * pp.kmax + k;
}

}  // namespace specgen
