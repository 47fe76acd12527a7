"""Nested prefixes (fork trees) on the GPU: fork-decode attention where a
fork attends over its trace's prefix chain, against the fp64 oracle."""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import check_attn, run_attn, sample_rows, say

pytestmark = pytest.mark.gpu

CASES = {
    # three nested trigger points; segments of 17, 1 and 31 tokens
    "chain3_tiny": dict(prefix_lens=[17, 1, 31], prefix_parent=[-1, 0, 1], forks_per_trace=[2, 1, 3],
                        suffix_lens=[0, 5, 16, 1, 0, 33], num_q_heads=8, num_kv_heads=2, head_dim=64),
    # two roots, branches, a grandchild; GQA 8 with up to 9 forks under a root
    "forest_mixed": dict(prefix_lens=[700, 300, 129, 64, 1500], prefix_parent=[-1, 0, 1, 0, -1],
                         forks_per_trace=[2, 3, 1, 2, 1], suffix_range=(0, 300), num_q_heads=16, num_kv_heads=2,
                         head_dim=128),
    # a chain of the maximum depth (8 traces), one fork per level
    "chain8": dict(prefix_lens=[100, 33, 16, 1, 250, 7, 64, 90], prefix_parent=[-1, 0, 1, 2, 3, 4, 5, 6],
                   forks_per_trace=1, suffix_range=(0, 40), num_q_heads=8, num_kv_heads=1, head_dim=64),
    # a root with no forks of its own: its prefix serves only the forks of the trace below it
    "empty_root": dict(prefix_lens=[64, 40], prefix_parent=[-1, 0], forks_per_trace=[0, 3],
                       suffix_lens=[0, 9, 33], num_q_heads=8, num_kv_heads=2, head_dim=128),
    # the shape of the nested workload, scaled down: 4 / 6 / 6 forks at three levels
    "chain3_gqa8": dict(prefix_lens=[2048, 1024, 1000], prefix_parent=[-1, 0, 1], forks_per_trace=[4, 6, 6],
                        suffix_range=(10, 200), num_q_heads=64, num_kv_heads=8, head_dim=128, key_bias_std=0.5),
}


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
@pytest.mark.parametrize("path", ["auto", "dot", "mfma"])
@pytest.mark.parametrize("name", list(CASES))
def test_tree_matches_oracle(name, path, kv):
    say(f"tree {name} path={path} kv={kv}")
    b = synth.make_fork_batch(kv_dtype=kv, seed=50 + list(CASES).index(name), **CASES[name])
    o, l = run_attn(b, path=path)
    ro, rl = oracle.fork_decode_attn(b)
    check_attn(o, ro, l, rl, what=f"{name} {path} {kv}")


def test_tree_equals_flat_batch_of_concatenated_prefixes():
    """A fork of the deepest level sees the same keys as a flat batch whose
    one prefix is the concatenation of the chain's segments (same pools, the
    chain's block tables joined when every segment but the last fills whole
    blocks)."""
    say("tree vs flat")
    b = synth.make_fork_batch(prefix_lens=[256, 512, 100], prefix_parent=[-1, 0, 1], forks_per_trace=[1, 1, 3],
                              suffix_lens=[4, 0, 17, 1, 60], num_q_heads=16, num_kv_heads=2, head_dim=128, seed=5)
    o, l = run_attn(b)
    import copy
    flat = copy.copy(b)
    flat.num_traces, flat.num_forks = 1, 3
    flat.fork_off = np.array([0, 3], np.int32)
    flat.prefix_len = np.array([int(b.prefix_len.sum())], np.int32)
    flat.prefix_table = np.ascontiguousarray(b.prefix_table)   # segments are whole blocks but the last
    flat.prefix_table_off = np.array([0, flat.prefix_table.size], np.int32)
    flat.suffix_len = b.suffix_len[2:].copy()
    flat.suffix_table_off = (b.suffix_table_off[2:] - b.suffix_table_off[2]).astype(np.int32)
    flat.suffix_table = b.suffix_table[b.suffix_table_off[2]:].copy()
    flat.q = b.q[2:].copy()
    flat.prefix_parent = None
    fo, fl = run_attn(flat)
    check_attn(o[2:], fo, l[2:], fl, what="tree vs flat")


def test_tree_full_size_sampled():
    """The nested workload at full size (segments of 16384, 8192 and 8192
    tokens; 4, 6 and 6 forks; 64 q heads over 8 kv heads), in the launch
    configuration the benchmark times, on 48 sampled rows."""
    say("tree full size tree_p32k_l3 sampled")
    b = synth.workload("tree_p32k_l3")
    o, l = run_attn(b)
    rows = sample_rows(b, 48, seed=2)
    ro, rl = oracle.fork_decode_attn(b, rows=rows)
    check_attn(o[rows[:, 0], rows[:, 1]], ro, l[rows[:, 0], rows[:, 1]], rl, what="tree_p32k_l3")
