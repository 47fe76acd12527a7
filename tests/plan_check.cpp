// plan_check.cpp -- CPU replay of the fork-decode work split.
//
// Builds plans for random batch shapes and unit prices with the host planner,
// then replays every worker's walk the way the attention kernels do (locate,
// segment lengths, segment index k) and every output row's merge lookup the way the
// merge kernel does, and checks:
//   - every tile of every work item is processed exactly once;
//   - per-worker item count and tile count stay within the kernels' caps;
//   - each row's merge finds exactly the (worker, segment) pairs that
//     processed its prefix items (one per trace on the fork's prefix chain,
//     for nested prefixes) and its suffix item, with in-range slots;
//   - each item row maps back to the (fork, q head) it belongs to;
//   - stepping from an item to the next (next_item) agrees with locate();
//   - per-worker units and tiles stay within the kernels' caps;
//   - the item table the walks record gives the merge the same workers and
//     slot index as the plan's own lookup.
// Built and run by tests/test_plan.py with g++ (no GPU involved).
#include <cstdio>
#include <cstdlib>
#include <algorithm>
#include <map>
#include <random>
#include <set>
#include <tuple>
#include <vector>

#include "../paper_2606_17518_amd/csrc/planner.h"

using namespace specgen;

#define CHECK(cond, ...)                                             \
  do {                                                               \
    if (!(cond)) {                                                   \
      fprintf(stderr, "FAIL %s:%d: %s | ", __FILE__, __LINE__, #cond); \
      fprintf(stderr, __VA_ARGS__);                                  \
      fprintf(stderr, "\n");                                         \
      return false;                                                  \
    }                                                                \
  } while (0)

struct Seg {
  int w, k;
  int64_t first;  // partition tile index of the segment's first tile
  int n;          // tiles
};

static int g_unsupported = 0;

// Forks of trace t and of every trace below it (nested prefixes), counted
// from the parent array directly: [fork_off[t], fork_off[e]) where e is the
// first later trace that does not descend from t.
static int subtree_rows(const PlanInputs& in, int t, int g) {
  int e = t + 1;
  for (; e < in.T; ++e) {
    int a = e;
    while (a >= 0 && a != t) a = in.prefix_parent ? in.prefix_parent[a] : -1;
    if (a != t) break;
  }
  return (in.fork_off[e] - in.fork_off[t]) * g;
}

// lib_prices: the library's unit prices, with which every generated shape
// must plan; with random prices the planner may answer "unsupported" (a
// range would touch more items than a kernel can describe), never wrongly.
static bool check_plan(const PlanInputs& in, int cus, uint64_t case_id, bool lib_prices) {
  Plan plan;
  int64_t wsf = 0;
  char err[256];
  const int rc = plan_build(in, [&] { return cus; }, &plan, &wsf, err, sizeof err);
  if (rc == kPlanUnsupported && !lib_prices) {
    ++g_unsupported;
    return true;
  }
  CHECK(rc == kPlanOk, "case %llu: plan_build failed: %s", (unsigned long long)case_id, err);
  // segments per (partition, item ordinal), from the walk the kernels run;
  // the walk also fills the item table the merge reads
  std::map<std::pair<int, int>, std::vector<Seg>> segs;
  std::vector<int32_t> tables[2];   // the item table of each partition (three int32 per item)
  for (int X = 0; X < 2; ++X) {
    const PartPlan& pp = plan.part[X];
    if (pp.workers == 0) {
      CHECK(pp.units == 0, "partition %d has units but no workers", X);
      continue;
    }
    CHECK(pp.info_base + 3 * (int64_t)pp.n_items <= wsf, "item table past the workspace");
    tables[X].assign(3 * (size_t)pp.n_items, -7);
    for (int w = 0; w < pp.workers; ++w) {
      const int64_t x0 = worker_start(pp, w), x1 = worker_start(pp, w + 1);

      int64_t x = x0;      // unit after the previous segment's last tile start
      int64_t data = 0;    // tiles visited so far
      bool fine = true;
      const WorkerRange wr = walk_range(plan, X, w, in.item_cap[X], [&](const ItemRef& it, int n, int rt, int i, int k) {
        const int64_t at = it.first + (int64_t)it.tile * it.w;   // unit where the segment's first tile starts
        // segments in order, inside the range (every tile start of a segment in
        // [x0, x1)), none before x0 missed
        if (it.kind < 0 || it.tile < 0 || n < 1 || it.tile + n > it.tiles || at < x || at < x0 ||
            at + (int64_t)(n - 1) * it.w >= x1 || (it.tile > 0 && at - it.w >= x0) || rt != data || k < 0 ||
            k >= pp.kmax || it.ord >= pp.n_items)
          fine = false;
        // the MFMA kernel stores whole 16-row N-tiles of an item's rows: the
        // rounded row count must fit the slot
        const int item_rows = std::min(it.kind == 0 ? trace_rows(plan, it.t) - it.rb * pp.rbs : plan.g - it.rb * pp.rbs,
                                       pp.rbs);
        if (item_rows < 1 || (X == kPartMfma ? (item_rows + 15) / 16 * 16 : item_rows) > pp.slot_rows) fine = false;
        segs[{X, it.ord}].push_back(Seg{w, k, at, n});
        if (it.ord >= 0 && it.ord < pp.n_items) record_item(tables[X].data(), it, n, w, k);
        x = at + (int64_t)(n - 1) * it.w + 1;
        data += n;
        (void)i;
      });
      CHECK(wr.R <= in.tile_cap[X], "worker %d holds %d tiles > cap", w, wr.R);
      CHECK(fine, "worker %d of partition %d: walk out of order or slot index out of range", w, X);
      // the chunked parallel walk of a partition that uses one must give the same segments
      if (in.walk_threads[X] > 0) {
        struct V { int ord, tile, n, rt, i, k; };
        std::vector<V> serial;
        walk_range(plan, X, w, in.item_cap[X], [&](const ItemRef& it, int n, int rt, int i, int k) {
          serial.push_back(V{it.ord, it.tile, n, rt, i, k});
        });
        std::vector<V> par;   // the parallel walk: one chunk of cu units per thread
        const int threads = in.walk_threads[X];
        const int cu = (int)((x1 - x0 + threads - 1) / threads);
        int first_ord = 0, ndata = 0;
        for (int tt = 0; tt < threads; ++tt) {
          const int64_t u0 = x0 + (int64_t)tt * cu;
          if (u0 >= x1) break;
          const TileInRange t = tile_in_chunk(plan, X, x0, x1, u0, cu);
          if (tt == 0) first_ord = t.it.ord;
          if (t.starts) par.push_back(V{t.it.ord, t.it.tile, t.n, ndata, (int)par.size(), t.it.ord - first_ord});
          ndata += t.data ? 1 : 0;
        }
        bool same = serial.size() == par.size();
        for (size_t q = 0; same && q < par.size(); ++q)
          same = serial[q].ord == par[q].ord && serial[q].tile == par[q].tile && serial[q].n == par[q].n &&
                 serial[q].rt == par[q].rt && serial[q].i == par[q].i && serial[q].k == par[q].k;
        CHECK(same, "worker %d of partition %d: chunked walk differs from the serial walk", w, X);
      }
      int64_t ndata = 0;   // tile starts in the range
      for (int64_t xx = x0; xx < x1; ++xx) {
        const ItemRef r = locate(plan, X, xx);
        ndata += (r.off >= 0 && r.off % r.w == 0) ? 1 : 0;
      }
      CHECK(wr.R == ndata, "worker %d walked %d of %lld data tiles (item cap %d)", w, wr.R, (long long)ndata,
            in.item_cap[X]);
    }
  }
  // enumerate items independently of locate() and check coverage
  const int g = in.Hq / in.Hkv;
  int64_t ptile[2] = {0, 0};
  int pord[2] = {0, 0};
  auto cover = [&](int X, int ord, int tiles, int wt, int charge) -> bool {
    auto itv = segs.find({X, ord});
    if (tiles == 0) {
      CHECK(itv == segs.end(), "empty item has segments");
      return true;
    }
    CHECK(itv != segs.end(), "item (%d, %d) never processed", X, ord);
    // an item takes `charge` units, then its tiles of wt units each
    int64_t expect = ptile[X] + charge;
    int total = 0;
    for (const Seg& s : itv->second) {
      CHECK(s.first == expect, "item tiles not contiguous");
      expect += (int64_t)s.n * wt;
      total += s.n;
    }
    CHECK(total == tiles, "item covered %d of %d tiles", total, tiles);
    ptile[X] += charge + (int64_t)tiles * wt;
    return true;
  };
  for (int X = 0; X < 2; ++X) {
    for (int t = 0; t < in.T; ++t) {
      const int rows = subtree_rows(in, t, g);
      if (part_of_trace(in.policy, rows) != X) continue;
      const int rb = (rows + in.rbs[X] - 1) / in.rbs[X];
      const int tiles = (in.prefix_len[t] + in.tt[X] - 1) / in.tt[X];
      for (int i = 0; i < in.Hkv * rb; ++i)
        if (!cover(X, pord[X]++, tiles, in.wt_rg[X][row_groups(std::min(rows, in.rbs[X]))], in.charge[X]))
          return false;
    }
  }
  {
    const int X = part_of_suffix(in.policy);
    const int rb = (g + in.rbs[X] - 1) / in.rbs[X];
    for (int f = 0; f < in.N; ++f) {
      const int tiles = (in.suffix_len[f] + in.tt[X] - 1) / in.tt[X];
      for (int i = 0; i < in.Hkv * rb; ++i)
        if (!cover(X, pord[X]++, tiles, in.wt_rg[X][row_groups(std::min(g, in.rbs[X]))], in.charge_suf[X]))
          return false;
    }
  }
  for (int X = 0; X < 2; ++X) CHECK(ptile[X] == plan.part[X].units, "partition %d unit total", X);
  // the incremental step between items agrees with locate() at every item boundary
  for (int X = 0; X < 2; ++X) {
    const PartPlan& pp = plan.part[X];
    int64_t x = 0;
    while (x < pp.units) {
      const ItemRef it = locate(plan, X, x);
      CHECK(it.off == -(it.kind == 0 ? pp.charge : pp.charge_suf), "an item starts with its charge");
      const int64_t nx = it.first + (int64_t)it.tiles * it.w;
      if (nx < pp.units) {
        const ItemRef a = next_item(plan, X, it);
        const int nc = nx >= pp.prefix_units ? pp.charge_suf : pp.charge;   // the next item's charge
        const ItemRef b = locate(plan, X, nx + nc);
        CHECK(a.kind == b.kind && a.t == b.t && a.f == b.f && a.j == b.j && a.rb == b.rb && a.tiles == b.tiles &&
                  a.tile == b.tile && a.off == b.off && a.w == b.w && a.first == b.first && a.ord == b.ord,
              "next_item differs from locate at unit %lld of partition %d", (long long)nx, X);
      }
      x = nx;
    }
  }
  // merge lookups
  auto same = [&](const ItemParts& ip, int ord) -> bool {
    const auto& v = segs.at({ip.part, ord});
    const int32_t* e = tables[ip.part].data() + 3 * (int64_t)ord;
    CHECK(e[0] == ip.w_lo && e[1] == ip.w_hi && e[2] == ip.k_lo, "item table (%d,%d,%d) vs parts (%d,%d,%d) at ord %d",
          e[0], e[1], e[2], ip.w_lo, ip.w_hi, ip.k_lo, ord);
    CHECK((int)v.size() == ip.w_hi - ip.w_lo + 1, "merge finds %d parts, %zu processed",
          ip.w_hi - ip.w_lo + 1, v.size());
    for (size_t i = 0; i < v.size(); ++i) {
      CHECK(v[i].w == ip.w_lo + (int)i, "worker mismatch");
      CHECK(v[i].k == (i == 0 ? ip.k_lo : 0), "segment index mismatch");
      const PartPlan& pp = plan.part[ip.part];
      const int64_t slot = slot_of(pp, v[i].w, v[i].k);
      CHECK(slot >= 0, "slot out of range");
      CHECK(part_o_off(pp, slot, ip.row + 1, in.D) <= pp.lse_base, "o slot past its region");
      CHECK(part_l_off(pp, slot, ip.row) + 2 <= pp.info_base, "lse slot past its region");
      CHECK(pp.info_base <= wsf, "regions past workspace");
      CHECK(ip.row >= 0 && ip.row < pp.slot_rows, "row in item");
    }
    return true;
  };
  const int parts_bound = max_parts_per_row(plan);   // what the merge launch sizes its batch for
  for (int f = 0; f < in.N; ++f) {
    int t = 0;
    while (in.fork_off[t + 1] <= f) ++t;
    CHECK(trace_of_fork(plan, f) == t, "trace_of_fork");
    std::vector<int> chain;   // the fork's own trace, then its ancestors
    for (int c = t; c >= 0; c = in.prefix_parent ? in.prefix_parent[c] : -1) chain.push_back(c);
    CHECK((int)chain.size() <= plan.depth, "chain of %zu traces, plan depth %d", chain.size(), plan.depth);
    for (int h = 0; h < in.Hq; ++h) {
      const int j = h / g, hh = h % g;
      int ff, hh2;
      int row_parts = 0;   // partials this row merges
      for (const int c : chain) {
        CHECK(plan.fork_off[c] <= f && f < plan.fork_end[c], "fork %d outside the rows of trace %d", f, c);
        const int ri = (f - in.fork_off[c]) * g + hh;
        const int X = plan.trace_part[c];
        const int rbs = in.rbs[X];
        const int rows = subtree_rows(in, c, g);
        const int rbc = (rows + rbs - 1) / rbs;
        // prefix item ordinal, counted directly
        int ord = 0;
        for (int t2 = 0; t2 < c; ++t2) {
          const int r2 = subtree_rows(in, t2, g);
          if (part_of_trace(in.policy, r2) == X) ord += in.Hkv * ((r2 + rbs - 1) / rbs);
        }
        ord += j * rbc + ri / rbs;
        const ItemParts P = prefix_parts_of_row(plan, f, h, c);
        CHECK(P.part == X, "prefix partition");
        {
          int xp = -1, op = -1, rp = -1;
          prefix_item_of_row(plan, f, h, c, &xp, &op, &rp);
          CHECK(xp == X && op == ord && rp == P.row, "prefix_item_of_row (%d,%d,%d) vs (%d,%d,%d)", xp, op, rp, X,
                ord, P.row);
          CHECK(op < plan.part[X].n_items, "prefix ordinal past the item table");
        }
        if (!same(P, ord)) return false;
        row_parts += P.w_hi - P.w_lo + 1;
        item_row_fork_head(plan, 0, c, -1, j, (ri / rbs) * rbs, P.row, &ff, &hh2);
        CHECK(ff == f && hh2 == h, "prefix row maps to (%d,%d) not (%d,%d)", ff, hh2, f, h);
      }
      ItemParts S;
      const bool has = suffix_parts_of_row(plan, f, h, &S);
      CHECK(has == (in.suffix_len[f] > 0), "suffix presence");
      if (!has) {
        int xs, os, rs;
        CHECK(!suffix_item_of_row(plan, f, h, &xs, &os, &rs), "suffix_item_of_row without suffix tokens");
      }
      if (has) {
        const int Xs = part_of_suffix(in.policy);
        const int rbss = in.rbs[Xs];
        const int srb = (g + rbss - 1) / rbss;
        const int sord = plan.part[Xs].n_prefix_items + (f * in.Hkv + j) * srb + hh / rbss;
        if (!same(S, sord)) return false;
        int xs = -1, os = -1, rs = -1;
        CHECK(suffix_item_of_row(plan, f, h, &xs, &os, &rs), "suffix_item_of_row presence");
        CHECK(xs == Xs && os == sord && rs == S.row, "suffix_item_of_row (%d,%d,%d) vs (%d,%d,%d)", xs, os, rs, Xs,
              sord, S.row);
        CHECK(os < plan.part[Xs].n_items, "suffix ordinal past the item table");
        CHECK(plan.part[Xs].info_base + 3 * (int64_t)plan.part[Xs].n_items <= wsf, "item table past workspace");
        item_row_fork_head(plan, 1, t, f, j, (hh / rbss) * rbss, S.row, &ff, &hh2);
        CHECK(ff == f && hh2 == h, "suffix row maps to (%d,%d) not (%d,%d)", ff, hh2, f, h);
        row_parts += S.w_hi - S.w_lo + 1;
      }
      CHECK(row_parts <= parts_bound, "row (%d,%d) merges %d parts, above the plan's bound %d", f, h, row_parts,
            parts_bound);
    }
  }
  return true;
}

int main(int argc, char** argv) {
  const int cases = argc > 1 ? atoi(argv[1]) : 300;
  const uint64_t seed = argc > 2 ? strtoull(argv[2], nullptr, 10) : 1;
  std::mt19937_64 rng(seed);
  auto U = [&](int lo, int hi) { return (int)(lo + rng() % (uint64_t)(hi - lo + 1)); };
  int done = 0;
  for (int c = 0; c < cases; ++c) {
    PlanInputs in;
    in.D = U(0, 1) ? 128 : 64;
    in.policy = U(0, 2);
    const int gs[] = {1, 2, 4, 8, 16, 24, 128};
    const int g = gs[U(0, 6)];
    in.Hkv = U(1, 3) == 1 ? 8 : U(1, 4);
    in.Hq = g * in.Hkv;
    // up to the per-call limits: a fifth of the cases have 13-32 traces, and a
    // tenth exactly 512 forks spread over the traces
    in.T = U(0, 4) == 0 ? U(13, kMaxTraces) : U(1, 12);
    std::vector<int32_t> fo(in.T + 1, 0), P(in.T);
    const bool most_forks = U(0, 9) == 0;
    for (int t = 0; t < in.T; ++t)
      fo[t + 1] = most_forks ? (int32_t)((t + 1) * (int64_t)kMaxForks / in.T) : fo[t] + U(1, U(0, 3) == 0 ? 40 : 6);
    in.N = fo[in.T];
    if (in.N > kMaxForks) continue;
    const int pmax = U(0, 4) == 0 ? 140000 : (U(0, 1) ? 3000 : 300);
    for (int t = 0; t < in.T; ++t) P[t] = U(1, pmax);
    std::vector<int32_t> S(in.N);
    const int smax = U(0, 1) ? 2100 : 40;
    for (int f = 0; f < in.N; ++f) S[f] = U(0, 3) == 0 ? 0 : U(0, smax);
    std::vector<int32_t> pto(in.T + 1, 0), sto(in.N + 1, 0);
    for (int t = 0; t < in.T; ++t) pto[t + 1] = pto[t] + (P[t] + 15) / 16;
    for (int f = 0; f < in.N; ++f) sto[f + 1] = sto[f] + (S[f] + 15) / 16;
    // nested prefixes in a third of the cases: a random depth-first forest of
    // depth <= kMaxDepth (each trace's parent is the previous trace or one of
    // its ancestors)
    std::vector<int32_t> parent(in.T, -1), depth(in.T, 1);
    const bool nested = U(0, 2) == 0;
    if (nested) {
      for (int t = 1; t < in.T; ++t) {
        int a = t - 1;
        const int up = U(0, 3);   // how many levels above the previous trace
        for (int k = 0; k < up && a >= 0; ++k) a = parent[a];
        if (a >= 0 && depth[a] >= kMaxDepth) a = parent[a];
        parent[t] = a;
        depth[t] = a < 0 ? 1 : depth[a] + 1;
      }
    }
    in.prefix_parent = nested ? parent.data() : nullptr;
    in.prefix_in_suffix_table = nullptr;
    in.fork_off = fo.data();
    in.prefix_len = P.data();
    in.suffix_len = S.data();
    in.prefix_table_off = pto.data();
    in.suffix_table_off = sto.data();
    in.tt[0] = in.D == 128 ? 64 : 128;
    in.tt[1] = 64;
    in.rbs[0] = 256;
    in.rbs[1] = 16;
    in.item_cap[0] = in.item_cap[1] = 64;
    // unit prices: the library's (bf16 or E4M3 MFMA prices and charges, dot
    // 1 / 1) or random; any positive prices must give a valid split
    const bool lib_prices = U(0, 1) != 0;
    if (lib_prices) {
      const bool e4m3 = U(0, 1) != 0;
      const int rg_bf16[9] = {0, 7, 7, 7, 8, 10, 11, 12, 13};
      const int rg_e4m3[9] = {0, 6, 6, 7, 8, 9, 10, 10, 11};
      for (int r = 0; r < 9; ++r) { in.wt_rg[0][r] = e4m3 ? rg_e4m3[r] : rg_bf16[r]; in.wt_rg[1][r] = 1; }
      in.charge[0] = e4m3 ? 16 : 20;
      in.charge[1] = 1;
      in.charge_suf[0] = e4m3 ? 16 : 12;
      in.charge_suf[1] = 1;
    } else {
      for (int X = 0; X < 2; ++X) {
        for (int r = 0; r < 9; ++r) in.wt_rg[X][r] = U(1, 16);
        in.charge[X] = U(0, 20);
        in.charge_suf[X] = U(0, 20);
      }
    }
    in.tile_cap[0] = 2560 / (in.tt[0] / 16);
    in.tile_cap[1] = 2048 / 4;
    in.walk_threads[0] = 512;   // the MFMA kernel's chunked walk
    in.walk_threads[1] = 0;     // the dot kernel's serial walk
    const int cus = U(0, 2) == 0 ? U(1, 16) : 256;
    if (!check_plan(in, cus, (uint64_t)c, lib_prices)) {
      fprintf(stderr, "case %d: D=%d policy=%d g=%d Hkv=%d T=%d N=%d cus=%d\n", c, in.D, in.policy, g, in.Hkv,
              in.T, in.N, cus);
      return 1;
    }
    ++done;
  }
  printf("OK %d plans (%d with random prices unsupported)\n", done, g_unsupported);
  return 0;
}
