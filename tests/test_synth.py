"""The seeded generator: reproducible, distinct block ids, poisoned unused slots."""
import numpy as np

import synth


def test_same_seed_same_bytes():
    a = synth.workload("tiny_p256_f4")
    b = synth.workload("tiny_p256_f4")
    for name in ("q", "k_pool", "v_pool", "prefix_table", "suffix_table", "suffix_len"):
        assert np.array_equal(getattr(a, name), getattr(b, name), equal_nan=False) or \
            np.array_equal(getattr(a, name).view(np.uint8), getattr(b, name).view(np.uint8))


def test_tables_are_distinct_and_in_range():
    b = synth.make_fork_batch(prefix_lens=[100, 33], forks_per_trace=[3, 2], suffix_range=(0, 40), num_q_heads=4,
                              num_kv_heads=2, head_dim=16, seed=7)
    ids = np.concatenate([b.prefix_table, b.suffix_table])
    assert len(np.unique(ids)) == len(ids)
    assert ids.min() >= 0 and ids.max() < b.num_blocks
    for t in range(b.num_traces):
        assert b.prefix_table_off[t + 1] - b.prefix_table_off[t] == -(-b.prefix_len[t] // 16)
    for f in range(b.num_forks):
        assert b.suffix_table_off[f + 1] - b.suffix_table_off[f] == -(-b.suffix_len[f] // 16)
        assert 0 <= b.suffix_len[f] <= 40


def test_unused_slots_are_nan_and_used_slots_finite():
    b = synth.make_fork_batch(prefix_lens=[21], forks_per_trace=2, suffix_lens=[0, 5], num_q_heads=2,
                              num_kv_heads=1, head_dim=8, seed=8)
    as_f32 = (b.k_pool.astype(np.uint32) << 16).view(np.float32)
    kf = np.isnan(as_f32).transpose(0, 2, 1, 3)            # K [NB][Hkv][16][D] -> [NB][16][Hkv][D]
    vf = np.isnan((b.v_pool.astype(np.uint32) << 16).view(np.float32)).transpose(0, 3, 1, 2)  # V [NB][Hkv][D][16]
    used = np.zeros((b.num_blocks, 16), bool)
    pt = b.prefix_table
    used[pt[0], :16] = True
    used[pt[1], :5] = True
    st = b.suffix_table
    used[st[0], :5] = True
    assert np.all(~kf[used]) and np.all(~vf[used])
    assert np.all(kf[~used]) and np.all(vf[~used])


def test_fp8_scales_positive_on_used_blocks():
    b = synth.make_fork_batch(prefix_lens=[40], forks_per_trace=1, suffix_lens=[10], num_q_heads=2,
                              num_kv_heads=1, head_dim=8, kv_dtype="fp8_e4m3", seed=9)
    ids = np.concatenate([b.prefix_table, b.suffix_table])
    assert np.all(b.k_scale[ids] > 0) and np.all(b.v_scale[ids] > 0)
    unused = np.setdiff1d(np.arange(b.num_blocks), ids)
    assert np.all(np.isnan(b.k_scale[unused]))
    # no NaN code in used slots
    assert not np.any(b.k_pool[b.prefix_table[0]] == 0x7F)
