// worker.h -- the part of a worker (workgroup) that both attention kernels
// share: list the items its tile range touches (with their lengths and table
// offsets, from the plan in LDS), and gather the block id of every 16-token
// block the range reads.  Everything lands in LDS so the tile loop never
// waits on a dependent load.
#pragma once
#include "common.h"
#include "plan.h"

namespace specgen {

// item descriptor fields (ints in LDS)
enum {
  IT_KIND, IT_T, IT_F, IT_J, IT_RB, IT_ORD, IT_TILE0, IT_NTILE, IT_NVALID, IT_TABOFF,
  IT_NROWS, IT_ROW0, IT_RTILE0, IT_TILES, IT_LASTBLK, IT_COUNT
};
constexpr int kItemInts = 16;
static_assert(IT_COUNT <= kItemInts, "item descriptor size");

// The item walk of a worker's tile range: every thread computes the same
// WorkerRange; thread 0 writes one descriptor per item into `items` (at most
// kItemCap; the host sizes workers so the cap holds).  It also records, in
// the partition's item table `info` (three int32 per item ordinal), which
// worker starts the item and its segment index there, and which worker ends
// it, so the merge finds an item's partials with one load.  No barrier at the
// end.
template <int kItemCap>
__device__ WorkerRange worker_walk(const Plan& plan, int part, int w, int32_t* items, int32_t* info) {
  const PartPlan& pp = plan.part[part];
  return walk_range(plan, part, w, kItemCap, [&](const ItemRef& it, int n, int rt, int i, int k) {
    if (threadIdx.x != 0) return;
    int32_t* d = items + i * kItemInts;
    d[IT_KIND] = it.kind;
    d[IT_T] = it.t;
    d[IT_F] = it.f;
    d[IT_J] = it.j;
    d[IT_RB] = it.rb;
    d[IT_ORD] = it.ord;
    d[IT_TILE0] = it.tile;
    d[IT_NTILE] = n;
    d[IT_RTILE0] = rt;
    d[IT_TILES] = it.tiles;
    const int r0 = it.rb * pp.rbs;
    const int rows = it.kind == 0 ? trace_rows(plan, it.t) : plan.g;
    d[IT_NROWS] = (rows - r0) < pp.rbs ? (rows - r0) : pp.rbs;
    d[IT_ROW0] = r0;
    const int nv = it.kind == 0 ? plan.prefix_len[it.t] : plan.suffix_len[it.f];
    d[IT_NVALID] = nv;
    d[IT_TABOFF] = it.kind == 0 ? plan.prefix_table_off[it.t] : plan.suffix_table_off[it.f];
    d[IT_LASTBLK] = (nv - 1) / 16;
    record_item(info, it, n, w, k);
  });
}

// The walk and the block-id gather in one pass: thread i examines the chunk
// of c = ceil((x1 - x0) / kThreads) units at x0 + i * c (tile_in_chunk; the
// planner keeps c within every tile price and the charge); a chunk where a
// tile starts loads the tile's kIdsPerTile block ids (clamped to its item's
// last valid block) into ids[n * kIdsPerTile ..], where n counts the tiles
// before it, and the thread at the first tile of each item's segment writes
// the item's descriptor and its item-table entries.  Items and tiles are
// numbered with wave ballots, so nothing runs serially and the only memory
// round trip is the id loads.  `scratch` is 2 * kThreads / 64 + 1 ints of
// LDS.  Ends with a barrier.
template <int kThreads, int kItemCap, int kIdsPerTile>
__device__ WorkerRange worker_walk_tiles(const AttnArgs& a, const Plan& plan, int part, int w, int32_t* items,
                                         int32_t* ids, int32_t* scratch) {
  constexpr int kW = kThreads / 64;
  const PartPlan& pp = plan.part[part];
  int32_t* info = reinterpret_cast<int32_t*>(a.ws + pp.info_base);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t x0 = worker_start(pp, w), x1 = worker_start(pp, w + 1);
  const int cu = (int)((x1 - x0 + kThreads - 1) / kThreads);   // units per chunk
  const int64_t u0 = x0 + (int64_t)tid * cu;
  const bool mine = u0 < x1;
  TileInRange tr;
  tr.data = tr.starts = false;
  tr.n = 0;
  int32_t id[kIdsPerTile];
  if (mine) {
    tr = tile_in_chunk(plan, part, x0, x1, u0, cu);
    if (tr.data) {
      const ItemRef& it = tr.it;
      const int nv = it.kind == 0 ? plan.prefix_len[it.t] : plan.suffix_len[it.f];
      const int lastblk = (nv - 1) / 16;
      const int32_t* tab = it.kind == 0 ? (plan.ptab_sel[it.t] ? a.suffix_table : a.prefix_table) +
                                              plan.prefix_table_off[it.t]
                                        : a.suffix_table + plan.suffix_table_off[it.f];
#pragma unroll
      for (int b = 0; b < kIdsPerTile; ++b) {
        const int bi = it.tile * kIdsPerTile + b;
        id[b] = tab[bi < lastblk ? bi : lastblk];
      }
    }
  }
  const uint64_t starts = __ballot(tr.starts);
  const uint64_t data = __ballot(tr.data);
  if (lane == 0) {
    scratch[wave] = __popcll(starts);
    scratch[kW + wave] = __popcll(data);
  }
  if (tid == 0) scratch[2 * kW] = mine ? tr.it.ord : 0;
  __syncthreads();
  int ibase = 0, items_total = 0, dbase = 0, data_total = 0;
#pragma unroll
  for (int v = 0; v < kW; ++v) {
    ibase += v < wave ? scratch[v] : 0;
    items_total += scratch[v];
    dbase += v < wave ? scratch[kW + v] : 0;
    data_total += scratch[kW + v];
  }
  const int first_ord = scratch[2 * kW];
  const uint64_t below = (1ull << lane) - 1;
  const int c = dbase + __popcll(data & below);   // data tiles before this one
  if (tr.starts) {
    const int i = ibase + __popcll(starts & below);
    if (i < kItemCap) {
      const ItemRef& it = tr.it;
      int32_t* d = items + i * kItemInts;
      d[IT_KIND] = it.kind;
      d[IT_T] = it.t;
      d[IT_F] = it.f;
      d[IT_J] = it.j;
      d[IT_RB] = it.rb;
      d[IT_ORD] = it.ord;
      d[IT_TILE0] = it.tile;
      d[IT_NTILE] = tr.n;
      d[IT_RTILE0] = c;
      d[IT_TILES] = it.tiles;
      const int r0 = it.rb * pp.rbs;
      const int rows = it.kind == 0 ? trace_rows(plan, it.t) : plan.g;
      d[IT_NROWS] = (rows - r0) < pp.rbs ? (rows - r0) : pp.rbs;
      d[IT_ROW0] = r0;
      const int nv = it.kind == 0 ? plan.prefix_len[it.t] : plan.suffix_len[it.f];
      d[IT_NVALID] = nv;
      d[IT_TABOFF] = it.kind == 0 ? plan.prefix_table_off[it.t] : plan.suffix_table_off[it.f];
      d[IT_LASTBLK] = (nv - 1) / 16;
      record_item(info, it, tr.n, w, it.ord - first_ord);
    }
  }
  if (tr.data) {
#pragma unroll
    for (int b = 0; b < kIdsPerTile; ++b) ids[c * kIdsPerTile + b] = id[b];
  }
  __syncthreads();
  WorkerRange wr;
  wr.nitems = items_total < kItemCap ? items_total : kItemCap;
  wr.first_ord = first_ord;
  wr.R = data_total;
  return wr;
}

// All threads of the block call this; `items` holds item_cap descriptors and
// `ids` holds tile_cap * ids_per_tile block ids.
// If `scales` is not null (E4M3 KV), scales[e] / scales[cap + e] receive the
// k / v block scale of ids[e], where cap = tile_cap * ids_per_tile.
template <int kThreads, int kItemCap, int kIdsPerTile, int kTileCap>
__device__ WorkerRange worker_prepass(const AttnArgs& a, const Plan& plan, int part, int w, int32_t* items,
                                      int32_t* ids, float* scales = nullptr) {
  const int tid = threadIdx.x;
  WorkerRange wr = worker_walk<kItemCap>(plan, part, w, items,
                                         reinterpret_cast<int32_t*>(a.ws + plan.part[part].info_base));
  if (wr.R <= 0) return wr;
  const int rt = wr.R;
  // the host sizes workers so the caps hold; never index past them
  wr.R = rt < kTileCap ? rt : kTileCap;
  __syncthreads();
  // 2. block ids of every tile of the range, clamped to the item's last valid block
  for (int e = tid; e < wr.R * kIdsPerTile; e += kThreads) {
    const int r = e / kIdsPerTile;
    const int b = e % kIdsPerTile;
    int ii = 0;
    while (ii + 1 < wr.nitems && items[(ii + 1) * kItemInts + IT_RTILE0] <= r) ++ii;
    const int32_t* d = items + ii * kItemInts;
    int bi = (d[IT_TILE0] + (r - d[IT_RTILE0])) * kIdsPerTile + b;
    if (bi > d[IT_LASTBLK]) bi = d[IT_LASTBLK];
    const int32_t* tab = (d[IT_KIND] == 0 && !plan.ptab_sel[d[IT_T]]) ? a.prefix_table : a.suffix_table;
    const int id = tab[d[IT_TABOFF] + bi];
    ids[e] = id;
    if (scales) {
      scales[e] = a.k_scale[id];
      scales[kTileCap * kIdsPerTile + e] = a.v_scale[id];
    }
  }
  __syncthreads();
  return wr;
}

// Index of the item that range tile r belongs to.
__device__ __forceinline__ int item_of_tile(const int32_t* items, int nitems, int r) {
  int ii = 0;
  while (ii + 1 < nitems && items[(ii + 1) * kItemInts + IT_RTILE0] <= r) ++ii;
  return ii;
}

// (fork, q head) of row rr of the item described by d.
__device__ __forceinline__ void item_row(const Plan& plan, const int32_t* d, int rr, int* fork, int* head) {
  item_row_fork_head(plan, d[IT_KIND], d[IT_T], d[IT_F], d[IT_J], d[IT_ROW0], rr, fork, head);
}

}  // namespace specgen
