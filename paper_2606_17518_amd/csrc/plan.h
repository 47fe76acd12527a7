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
// `tt` tokens.  In the partition's tile sequence every item is preceded by
// `charge` empty tiles: they stand for the item's fixed cost in a worker (its
// query rows and its end), so workers whose ranges hold many short items get
// fewer tiles of data.  The sequence is split evenly over W workers
// (workgroups): worker w takes positions [start(w), start(w+1)) and processes
// the real tiles among them.  A worker emits
// one partial (o, lse) per item it touches, into slot w * kmax + k where k is
// the item's ordinal minus the ordinal of the worker's first item.  The merge
// finds the workers covering an item from its tile range alone.
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
constexpr int kBlock = 16;       // tokens per KV block

enum { kPartMfma = 0, kPartDot = 1 };
enum { kPolicyAuto = 0, kPolicyDot = 1, kPolicyMfma = 2 };

struct PartPlan {
  int64_t tiles;          // total tiles of the partition
  int64_t prefix_tiles;   // tiles of its prefix items (they come first)
  int64_t o_base;         // float offset of slot 0's o (fp16 rows, see part_row_k) in the workspace
  int64_t lse_base;       // float offset of slot 0's (lse, dec) pairs
  int64_t info_base;      // float offset of the item table: per item ordinal three
                          // int32 (first worker, last worker, segment index in the first)
  int32_t n_items;        // items of the partition (prefix, then suffix)
  int32_t per_lo;         // tiles / W: every worker gets per_lo tiles, the first
  int32_t n_hi;           // tiles % W workers one more
  int32_t workers;        // W (0: partition unused)
  int32_t kmax;           // max items touched by one worker
  int32_t tt;             // tokens per tile
  int32_t rbs;            // rows per row block
  int32_t slot_rows;      // rows reserved per partial slot (== rbs)
  int32_t n_prefix_items; // prefix items in the partition
  int32_t has_suffix;     // suffix items belong to this partition
  int32_t suffix_rb;      // row blocks per suffix (fork, head): ceil(g / rbs)
  int32_t n_traces;       // traces whose prefix items are in the partition
  int32_t trace_begin;    // their positions in Plan::ptrace: [trace_begin, +n_traces)
  int32_t charge;         // empty tiles in front of every item
};

// The scalar part of the plan.
struct PlanHead {
  int32_t T, N, Hq, Hkv, g, D;
  int32_t policy, pad_;
  PartPlan part[2];
};

// The whole plan, computed on the host from the length mirrors and passed to
// every kernel by value (about 7.3 KB of kernel arguments); each workgroup
// copies it into LDS with one vector load per thread (plan_to_lds).
struct alignas(16) Plan : PlanHead {
  int32_t fork_off[kMaxTraces + 1];
  int32_t prefix_len[kMaxTraces];
  int32_t trace_part[kMaxTraces];   // partition of trace t's prefix items
  int32_t trace_pos[kMaxTraces];    // index of t in ptrace
  int32_t ptrace[kMaxTraces];       // traces grouped by partition, ascending within each
  int32_t tileP[kMaxTraces];        // (by ptrace position) first tile of the trace's prefix items
  int32_t ordP[kMaxTraces];         // (by ptrace position) ordinal of its first prefix item
  int32_t tileS[kMaxForks + 1];     // first tile of fork f's suffix items, relative to prefix_tiles
  int32_t prefix_table_off[kMaxTraces + 1];   // host mirrors of the batch's index arrays
  int32_t suffix_len[kMaxForks];
  int32_t suffix_table_off[kMaxForks + 1];
};

SG_HD int32_t cdiv(int64_t a, int64_t b) { return (int32_t)((a + b - 1) / b); }
SG_HD int32_t cdiv32(int32_t a, int32_t b) { return (a + b - 1) / b; }



SG_HD int32_t trace_rows(const Plan& p, int t) { return (p.fork_off[t + 1] - p.fork_off[t]) * p.g; }

SG_HD int part_of_trace(int policy, int rows) {
  if (policy == kPolicyDot) return kPartDot;
  if (policy == kPolicyMfma) return kPartMfma;
  return rows >= 16 ? kPartMfma : kPartDot;
}

SG_HD int part_of_suffix(int policy) { return policy == kPolicyDot ? kPartDot : kPartMfma; }

// First tile of worker w: workers [0, n_hi) take per_lo + 1 tiles, the rest
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

// Worker owning tile x: the largest w with worker_start(w) <= x.
// Tile positions fit in 32 bits (the planner rejects larger partitions), so
// the divisions are 32-bit.
SG_HD int32_t worker_of_tile(const PartPlan& pp, int64_t x) {
  const uint32_t big = (uint32_t)pp.n_hi * (uint32_t)(pp.per_lo + 1);   // tiles of the larger ranges
  const uint32_t xx = (uint32_t)x;
  if (xx < big) return (int32_t)(xx / (uint32_t)(pp.per_lo + 1));
  return (int32_t)((uint32_t)pp.n_hi + (xx - big) / (uint32_t)pp.per_lo);
}

struct ItemRef {
  int32_t kind;      // 0 prefix, 1 suffix, -1 past the end
  int32_t t, f, j, rb;
  int32_t tiles;     // tiles of the item (its data)
  int32_t tile;      // tile of x within the item; -charge..-1 for its empty tiles
  int64_t first;     // sequence position of the item's first tile of data
  int32_t ord;       // ordinal of the item in the partition
};

// Sequence positions taken by one suffix item of fork f (0 if S_f = 0): its
// charge plus ceil(S_f / tt); tileS holds their per-fork prefix sums.
SG_HD int32_t suffix_span(const Plan& p, const PartPlan& pp, int f) {
  return (p.tileS[f + 1] - p.tileS[f]) / (p.Hkv * pp.suffix_rb);
}

// The item at partition sequence position x.
SG_HD ItemRef locate(const Plan& p, int part, int64_t x) {
  const PartPlan& pp = p.part[part];
  ItemRef r;
  r.kind = -1;
  r.t = r.f = r.j = r.rb = r.tiles = r.tile = r.ord = 0;
  r.first = 0;
  if (x < 0 || x >= pp.tiles) return r;
  if (x < pp.prefix_tiles) {
    // largest position i in the partition's trace list with tileP[i] <= x
    int lo = pp.trace_begin, hi = pp.trace_begin + pp.n_traces - 1;
    while (lo < hi) {
      int mid = (lo + hi + 1) >> 1;
      if (p.tileP[mid] <= x) lo = mid; else hi = mid - 1;
    }
    const int t = p.ptrace[lo];
    const int rb_count = cdiv32(trace_rows(p, t), pp.rbs);
    const int tiles = cdiv32(p.prefix_len[t], pp.tt);
    const int span = tiles + pp.charge;
    const int local = (int)(x - p.tileP[lo]);   // tile counts fit in int32 (the planner checks)
    const int item = local / span;
    r.kind = 0;
    r.t = t;
    r.j = item / rb_count;
    r.rb = item % rb_count;
    r.tiles = tiles;
    r.tile = local - item * span - pp.charge;
    r.first = x - r.tile;
    r.ord = p.ordP[lo] + item;
    return r;
  }
  const int xs = (int)(x - pp.prefix_tiles);
  int lo = 0, hi = p.N - 1;   // largest f with tileS[f] <= xs
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (p.tileS[mid] <= xs) lo = mid; else hi = mid - 1;
  }
  const int f = lo;
  const int span = suffix_span(p, pp, f);
  const int local = xs - p.tileS[f];
  const int item = local / span;
  r.kind = 1;
  r.f = f;
  r.j = item / pp.suffix_rb;
  r.rb = item % pp.suffix_rb;
  r.tiles = span - pp.charge;
  r.tile = local - item * span - pp.charge;
  r.first = x - r.tile;
  r.ord = pp.n_prefix_items + (f * p.Hkv + r.j) * pp.suffix_rb + r.rb;
  return r;
}

// The item that follows `cur` in partition `part` (cur must not be the last
// one), at its first tile of data: equal to
// locate(p, part, cur.first + cur.tiles + charge).  Steps within a trace or
// fork in O(1) and falls back to locate() where it would have to skip over
// forks without suffix tokens or cross into the suffix items.
SG_HD ItemRef next_item(const Plan& p, int part, const ItemRef& cur) {
  const PartPlan& pp = p.part[part];
  const int64_t x = cur.first + cur.tiles + pp.charge;
  ItemRef r = cur;
  r.first = x;
  r.tile = 0;
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
      return r;
    }
    return locate(p, part, x);
  }
  if (cur.rb + 1 < pp.suffix_rb) {
    r.rb = cur.rb + 1;
    return r;
  }
  if (cur.j + 1 < p.Hkv) {
    r.j = cur.j + 1;
    r.rb = 0;
    return r;
  }
  const int f = cur.f + 1;
  if (f < p.N) {
    const int tiles = suffix_span(p, pp, f) - pp.charge;
    if (tiles > 0) {
      r.f = f;
      r.j = 0;
      r.rb = 0;
      r.tiles = tiles;
      return r;
    }
  }
  return locate(p, part, x);
}

// The items of worker w's range, in order.  For each one with tiles of data
// in the range calls visit(it, n, rt, i, k): it = the item (it.tile = its
// first tile in the range), n = its tiles in the range, rt = the number of
// data tiles of the range before them (empty tiles do not count), i = its
// position among the visited items, k = it.ord - (ordinal of the item at the
// range's first position), which is the partial-slot index (w * kmax + k).
// At most item_cap items are visited.
struct WorkerRange {
  int nitems;     // items visited
  int first_ord;  // ordinal of the item at the range's first position
  int R;          // data tiles in the range
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
  int64_t x = x0;
  if (it.tile < 0) {   // the range starts on the item's empty tiles
    x = it.first;
    it.tile = 0;
  }
  while (x < x1 && wr.nitems < item_cap) {
    const int n = (int)((it.tiles - it.tile) < (x1 - x) ? (it.tiles - it.tile) : (x1 - x));
    visit(it, n, wr.R, wr.nitems, it.ord - wr.first_ord);
    wr.R += n;
    ++wr.nitems;
    x += n;
    if (x >= x1) break;
    it = next_item(p, part, it);
    x = it.first;   // past the next item's empty tiles
  }
  return wr;
}

// The parallel form of walk_range: what position x of worker w's range
// [x0, x1) contributes.  `data` marks a tile of data (not an item's empty
// tile); `starts` marks the first data tile of an item's segment in the range
// (x == x0 or the item's own first data tile); there, n is the segment's
// length.  The segments in order of x are exactly walk_range's visits: the
// visit index of a segment is the number of starting positions before it, its
// rt the number of data positions before it, and its slot index it.ord minus
// the ordinal of the item at x0.
struct TileInRange {
  ItemRef it;
  bool data;
  bool starts;
  int n;
};
SG_HD TileInRange tile_in_range(const Plan& p, int part, int64_t x0, int64_t x1, int64_t x) {
  TileInRange r;
  r.it = locate(p, part, x);
  r.data = r.it.tile >= 0;
  r.starts = r.data && (x == x0 || r.it.tile == 0);
  const int64_t left = x1 - x;
  const int rest = r.it.tiles - r.it.tile;
  r.n = rest < left ? rest : (int)left;
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

SG_HD ItemParts item_parts(const Plan& p, int part, int64_t first_tile, int tiles, int ord, int row) {
  const PartPlan& pp = p.part[part];
  ItemParts ip;
  ip.part = part;
  ip.row = row;
  ip.w_lo = worker_of_tile(pp, first_tile);
  ip.w_hi = worker_of_tile(pp, first_tile + tiles - 1);
  const ItemRef f0 = locate(p, part, worker_start(pp, ip.w_lo));
  ip.k_lo = ord - f0.ord;
  return ip;
}

// The prefix item of row (f, h) and its row inside the item.
SG_HD ItemParts prefix_parts_of_row(const Plan& p, int f, int h) {
  const int g = p.g, j = h / g, hh = h - j * g;
  const int t = trace_of_fork(p, f);
  const int ri = (f - p.fork_off[t]) * g + hh;
  const int X = p.trace_part[t];
  const PartPlan& pp = p.part[X];
  const int rbc = cdiv32(trace_rows(p, t), pp.rbs);
  const int rb = ri / pp.rbs;
  const int tiles = cdiv32(p.prefix_len[t], pp.tt);
  const int pos = p.trace_pos[t];
  const int item = j * rbc + rb;
  return item_parts(p, X, (int64_t)p.tileP[pos] + (int64_t)item * (tiles + pp.charge) + pp.charge, tiles,
                    p.ordP[pos] + item, ri - rb * pp.rbs);
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
  *out = item_parts(p, X, pp.prefix_tiles + p.tileS[f] + (int64_t)item * span + pp.charge, span - pp.charge,
                    pp.n_prefix_items + f * per_fork + item, hh - rb * pp.rbs);
  return true;
}

// The prefix item of row (f, h): its partition, ordinal and the row inside it.
SG_HD void prefix_item_of_row(const Plan& p, int f, int h, int* part, int* ord, int* row) {
  const int g = p.g, j = h / g, hh = h - j * g;
  const int t = trace_of_fork(p, f);
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
  if (p.tileS[f + 1] == p.tileS[f]) return false;
  const int rb = hh / pp.rbs;
  *part = X;
  *ord = pp.n_prefix_items + (f * p.Hkv + j) * pp.suffix_rb + rb;
  *row = hh - rb * pp.rbs;
  return true;
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
