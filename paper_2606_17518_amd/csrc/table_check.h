// table_check.h -- host-only check that every block id the attention kernels
// of a planned batch will read lies in [0, num_blocks).  The release library
// leaves that precondition to the caller (the tables are device memory and
// checking them costs a copy to the host and a synchronisation); the library
// built with SPECGEN_DEBUG_CHECKS runs this check before every launch.  Plain
// C++ with no HIP dependency, so a g++ test harness drives it with host
// tables.
#pragma once
#include <stdint.h>

#include <vector>

#include "plan.h"

namespace specgen {

enum { kTableOk = 0, kTableBadId = 1, kTableFetchFailed = 2 };

struct BadBlockId {
  int table;       // 0: prefix table, 1: suffix table
  int kind;        // the reader: 0, a trace's prefix; 1, a fork's suffix
  int owner;       // that trace or fork
  int64_t entry;   // index of the entry in its table
  int32_t id;      // the id found there
};

// The ids read are, for trace t, ceil(P_t / 16) entries from
// prefix_table_off[t] (of the suffix table where ptab_sel[t] is set) and, for
// fork f, ceil(S_f / 16) entries from suffix_table_off[f]; entries past those
// are never read and are not checked.  Each table's span of read entries is
// fetched once: fetch(table, first, count, dst) copies entries [first, first
// + count) of table 0 (prefix) or 1 (suffix) to dst and returns false on
// failure.  Returns kTableOk, kTableBadId (the first bad entry, traces before
// forks, in *bad) or kTableFetchFailed.
template <typename Fetch>
int check_block_ids(const Plan& p, int64_t num_blocks, Fetch fetch, BadBlockId* bad) {
  struct Range {
    int table, kind, owner;
    int64_t first, count;
  };
  std::vector<Range> ranges;
  for (int t = 0; t < p.T; ++t)
    ranges.push_back({p.ptab_sel[t] ? 1 : 0, 0, t, p.prefix_table_off[t], cdiv(p.prefix_len[t], kBlock)});
  for (int f = 0; f < p.N; ++f)
    if (p.suffix_len[f] > 0) ranges.push_back({1, 1, f, p.suffix_table_off[f], cdiv(p.suffix_len[f], kBlock)});
  int64_t lo[2] = {INT64_MAX, INT64_MAX}, hi[2] = {0, 0};
  for (const Range& r : ranges) {
    if (r.count <= 0) continue;
    lo[r.table] = r.first < lo[r.table] ? r.first : lo[r.table];
    hi[r.table] = r.first + r.count > hi[r.table] ? r.first + r.count : hi[r.table];
  }
  std::vector<int32_t> ids[2];
  for (int tb = 0; tb < 2; ++tb) {
    if (lo[tb] >= hi[tb]) continue;
    ids[tb].resize((size_t)(hi[tb] - lo[tb]));
    if (!fetch(tb, lo[tb], hi[tb] - lo[tb], ids[tb].data())) return kTableFetchFailed;
  }
  for (const Range& r : ranges) {
    for (int64_t i = 0; i < r.count; ++i) {
      const int32_t id = ids[r.table][(size_t)(r.first + i - lo[r.table])];
      if (id < 0 || (int64_t)id >= num_blocks) {
        *bad = BadBlockId{r.table, r.kind, r.owner, r.first + i, id};
        return kTableBadId;
      }
    }
  }
  return kTableOk;
}

}  // namespace specgen
