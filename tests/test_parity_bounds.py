"""The full-size lse bound can see a lost KV block (CPU only, oracle only).

The GPU parity tests bound |d lse| by 1e-4 on the full-size decode workloads,
beside the output tolerances.  Here the oracle shows why both are
needed: on rows shaped like the 32k-prefix workload (one kv head of it: a
32768-token prefix, 16 forks with 128-1024 suffix tokens, GQA group of 8,
D = 128, keys N(0, 1) plus a per-head bias of std 0.5), removing a single
16-token prefix block leaves the bf16-sized output change under the output
tolerances (the softmax over ~33k keys is nearly flat), but moves every
row's lse by several times 1e-4.
"""
import dataclasses

import numpy as np

import oracle
import synth
from gpu_helpers import ATTN_MAX_ABS, ATTN_MEAN_ABS, LSE_FULL_SIZE_MAX_ABS


def _drop_block(b, k):
    """The batch with prefix block k of trace 0 removed (every block is full)."""
    assert b.num_traces == 1 and b.prefix_len[0] % 16 == 0
    out = dataclasses.replace(b)
    out.prefix_table = np.delete(b.prefix_table, k).astype(np.int32)
    out.prefix_table_off = np.array([0, len(out.prefix_table)], np.int32)
    out.prefix_len = np.array([b.prefix_len[0] - 16], np.int32)
    return out


def test_dropped_prefix_block_breaks_the_full_size_lse_bound():
    b = synth.make_fork_batch(prefix_lens=[32768], forks_per_trace=16, suffix_range=(128, 1024), num_q_heads=8,
                              num_kv_heads=1, head_dim=128, key_bias_std=0.5, extra_blocks=0, seed=3)
    ref, ref_l = oracle.fork_decode_attn(b)
    for k in (0, 1000, 2047):
        out, lse = oracle.fork_decode_attn(_drop_block(b, k))
        d_out = np.abs(out - ref)
        d_lse = np.abs(lse - ref_l)
        # invisible to the output tolerances ...
        assert d_out.max() < ATTN_MAX_ABS and d_out.mean() < ATTN_MEAN_ABS
        # ... but every row's lse moves past the full-size bound, most by far
        assert d_lse.min() > LSE_FULL_SIZE_MAX_ABS, (k, d_lse.min())
        assert np.median(d_lse) > 3 * LSE_FULL_SIZE_MAX_ABS, (k, np.median(d_lse))
