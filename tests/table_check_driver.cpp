// Host harness of the debug build's block-id check (table_check.h): builds
// small plans by hand and checks which table entry the check reports.
#include <stdio.h>
#include <string.h>

#include <vector>

#include "../paper_2606_17518_amd/csrc/table_check.h"

using namespace specgen;

static int failures = 0;
#define EXPECT(c)                                              \
  do {                                                         \
    if (!(c)) {                                                \
      printf("FAILED line %d: %s\n", __LINE__, #c);            \
      ++failures;                                              \
    }                                                          \
  } while (0)

struct Tables {
  std::vector<int32_t> t[2];
  int fetches = 0;
  bool fail = false;
};

static int run(const Plan& p, int64_t num_blocks, Tables& tb, BadBlockId* bad) {
  auto fetch = [&](int table, int64_t first, int64_t count, int32_t* dst) {
    ++tb.fetches;
    if (tb.fail || first < 0 || first + count > (int64_t)tb.t[table].size()) return false;
    memcpy(dst, tb.t[table].data() + first, (size_t)count * 4);
    return true;
  };
  return check_block_ids(p, num_blocks, fetch, bad);
}

int main() {
  static Plan p;   // large: not on the stack
  memset(&p, 0, sizeof p);
  // two traces (P = 40, 16), three forks (S = 17, 0, 5); tables with spare
  // entries after each range, which hold out-of-range ids that are never read
  p.T = 2;
  p.N = 3;
  p.prefix_len[0] = 40;   // 3 ids at 0
  p.prefix_len[1] = 16;   // 1 id at 4
  p.prefix_table_off[0] = 0;
  p.prefix_table_off[1] = 4;
  p.prefix_table_off[2] = 6;
  p.suffix_len[0] = 17;   // 2 ids at 0
  p.suffix_len[1] = 0;    // none
  p.suffix_len[2] = 5;    // 1 id at 3
  p.suffix_table_off[0] = 0;
  p.suffix_table_off[1] = 3;
  p.suffix_table_off[2] = 3;
  p.suffix_table_off[3] = 5;
  const int64_t NB = 10;
  Tables tb;
  tb.t[0] = {0, 9, 2, -7, 5, 99};
  tb.t[1] = {3, 4, 1000, 8, -1};
  BadBlockId bad;
  EXPECT(run(p, NB, tb, &bad) == kTableOk);
  EXPECT(tb.fetches == 2);
  // num_blocks itself is out of range: id 9 in prefix entry 1
  EXPECT(run(p, 9, tb, &bad) == kTableBadId);
  EXPECT(bad.table == 0 && bad.kind == 0 && bad.owner == 0 && bad.entry == 1 && bad.id == 9);
  // -1 in the second trace's only id
  tb.t[0][4] = -1;
  EXPECT(run(p, NB, tb, &bad) == kTableBadId);
  EXPECT(bad.table == 0 && bad.owner == 1 && bad.entry == 4 && bad.id == -1);
  tb.t[0][4] = 5;
  // a bad id in the last suffix block of fork 0 (17 tokens: two blocks)
  tb.t[1][1] = 10;
  EXPECT(run(p, NB, tb, &bad) == kTableBadId);
  EXPECT(bad.table == 1 && bad.kind == 1 && bad.owner == 0 && bad.entry == 1 && bad.id == 10);
  tb.t[1][1] = 4;
  // fork 1 is empty: its range start (3) is fork 2's, whose id 8 is fine;
  // entry 2 (1000) belongs to nobody
  EXPECT(run(p, NB, tb, &bad) == kTableOk);
  // a longer suffix for fork 2 reads entry 4 (-1)
  p.suffix_len[2] = 20;
  EXPECT(run(p, NB, tb, &bad) == kTableBadId);
  EXPECT(bad.table == 1 && bad.owner == 2 && bad.entry == 4 && bad.id == -1);
  p.suffix_len[2] = 5;
  // a trace whose prefix ids live in the suffix table (prefill nesting)
  p.ptab_sel[1] = 1;
  p.prefix_table_off[1] = 2;   // suffix entry 2: 1000
  EXPECT(run(p, NB, tb, &bad) == kTableBadId);
  EXPECT(bad.table == 1 && bad.kind == 0 && bad.owner == 1 && bad.entry == 2 && bad.id == 1000);
  p.prefix_table_off[1] = 3;   // suffix entry 3: 8
  EXPECT(run(p, NB, tb, &bad) == kTableOk);
  // a failed read-back is reported as such
  tb.fail = true;
  EXPECT(run(p, NB, tb, &bad) == kTableFetchFailed);
  tb.fail = false;
  // every suffix empty and no trace in the suffix table: the suffix table is not read
  p.ptab_sel[1] = 0;
  p.prefix_table_off[1] = 4;
  for (int f = 0; f < 3; ++f) p.suffix_len[f] = 0;
  tb.t[1].clear();
  tb.fetches = 0;
  EXPECT(run(p, NB, tb, &bad) == kTableOk);
  EXPECT(tb.fetches == 1);
  if (failures) return 1;
  printf("all table checks passed\n");
  return 0;
}
