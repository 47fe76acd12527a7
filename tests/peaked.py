"""Peaked-attention inputs for the parity tests: queries that make each row's
softmax concentrate on a planted key placed relative to the key-axis split the
library reports (specgen_fork_decode_attn_split), so that

  - a dominant key sits at the first token of a workgroup's range (just after
    a boundary), three quarters into a range (after the range's running max is
    established, so the kernel must rescale mid-item), or on the last token
    of a range (just before a boundary), or in the fork's suffix;
  - every row's scores spread over well beyond 20 nats (queries scaled by
    q_scale), so the partial results span a wide dynamic range.

Only input construction lives here; the expected values come from the oracle."""
import numpy as np

import paper_2606_17518_amd as sg
from synth.fork_batch import with_peaked_queries

Q_SCALE = 2.5
CASES = ("boundary", "late", "before_boundary", "suffix", "none", "start")


def planted_positions(batch, path="auto"):
    """key_index [N][Hq] (-1: none), weight [N][Hq] and the case name of each row."""
    sp = sg.specgen_fork_decode_attn_split(batch, path)
    N, Hq, g = batch.num_forks, batch.num_q_heads, batch.group
    segs = {}   # (trace, kv head, row) -> sorted token ranges of the row's prefix item
    for k in np.flatnonzero(sp["kind"] == 0):
        t, j = int(sp["trace"][k]), int(sp["kv_head"][k])
        for r in range(int(sp["first_row"][k]), int(sp["first_row"][k] + sp["num_rows"][k])):
            segs.setdefault((t, j, r), []).append((int(sp["first_token"][k]), int(sp["num_tokens"][k])))
    key = np.full((N, Hq), -1, np.int64)
    weight = np.zeros((N, Hq), np.float32)
    case = np.empty((N, Hq), object)
    rng = np.random.default_rng(12345)
    for f in range(N):
        t = batch.trace_of_fork(f)
        assert batch.prefix_chain(t) == [t], "planting supports root traces only"
        P, S = int(batch.prefix_len[t]), int(batch.suffix_len[f])
        for h in range(Hq):
            row = (f - int(batch.fork_off[t])) * g + h % g
            ranges = sorted(segs[(t, h // g, row)])
            c = CASES[(f * Hq + h) % len(CASES)]
            if c == "suffix" and S == 0:
                c = "late"
            k = 1 + (f * 7 + h) % (len(ranges) - 1) if len(ranges) > 1 else 0
            first, n = ranges[k]
            if c == "boundary":
                key[f, h] = first
            elif c == "late":
                key[f, h] = first + (3 * n) // 4
            elif c == "before_boundary":
                key[f, h] = first + n - 1
            elif c == "suffix":
                key[f, h] = P + int(rng.integers(0, S))
            elif c == "start":
                key[f, h] = 0
            case[f, h] = c
            weight[f, h] = 2.0 if (f + h) % 2 == 0 else 1.0
    return key, weight, case


def peaked_batch(batch, path="auto"):
    key, weight, case = planted_positions(batch, path)
    return with_peaked_queries(batch, key, weight, Q_SCALE), case
