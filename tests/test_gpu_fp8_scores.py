"""E4M3 KV with fp8 scores (SPECGEN_FLAG_FP8_SCORES) on the GPU against the fp64 oracle.

The scores q . k run on the fp8 matrix cores from the K codes, with each query
row as two E4M3 terms; the oracle is the same plain definition over the
dequantised KV, so the bar is the same: max abs 1e-2 and mean abs 1e-3 on the
bf16 output, |d lse| <= 1e-3, and on the full-size 128k-prefix workload the lse
bound of 1e-4 that resolves a single 16-token block.  Peaked inputs (planted
dominant keys at the split boundaries, tests/peaked.py) use the tolerances on
the error beyond the bf16 output's own rounding.
"""
import numpy as np
import pytest

import oracle
import paper_2606_17518_amd as sg
import synth
from gpu_helpers import LSE_FULL_SIZE_MAX_ABS, check_attn, check_attn_excess, run_attn, sample_rows, say
from test_gpu_peaked import _check as peaked_check

pytestmark = pytest.mark.gpu
F8 = sg.SPECGEN_FLAG_FP8_SCORES

# (prefix lens, forks per trace, suffix lens, Hq, Hkv): E4M3, D = 128
SMALL = [
    ([300], 4, [0, 3, 33, 70], 16, 2),                      # r = 32
    ([500], 16, list(range(5, 165, 10)), 256, 16),          # r = 256: one token group per wave
    ([1], 1, [0], 8, 8),                                    # one key: out is its value row
    ([17], 2, [16, 1], 16, 1),                              # g = 16, r = 32
    ([65, 190], [2, 3], [1, 0, 16, 17, 80], 32, 8),         # two traces, r = 8 and 12 (dot path under auto)
    ([1000], 5, [7, 300, 0, 64, 129], 64, 8),               # r = 40
    ([130], 20, [1] * 20, 160, 8),                          # r = 400: row blocks of 256 and 144
]


@pytest.mark.parametrize("path", ["auto", "mfma"])
@pytest.mark.parametrize("i", range(len(SMALL)))
def test_small_shapes_all_rows(i, path):
    P, F, S, Hq, Hkv = SMALL[i]
    b = synth.make_fork_batch(prefix_lens=P, forks_per_trace=F, suffix_lens=S, num_q_heads=Hq, num_kv_heads=Hkv,
                              head_dim=128, kv_dtype="fp8_e4m3", seed=400 + i)
    say(f"fp8 scores small {i} {path}")
    ref, ref_l = oracle.fork_decode_attn(b)
    out, lse = run_attn(b, path, flags=F8)
    if sum(P) + max(S) == 1:
        # one key: the output is that key's value row (E4M3 code x block scale, of
        # order one), which the bf16 output rounds by up to 2^-8 of itself
        check_attn_excess(out, ref, lse, ref_l, what=f"fp8 scores small {i} {path}")
    else:
        check_attn(out, ref, lse, ref_l, what=f"fp8 scores small {i} {path}")


def test_full_size_128k_prefix():
    say("fp8_p128k_f32: generating")
    b = synth.workload("fp8_p128k_f32")
    rows = sample_rows(b, 256, seed=8)
    ref, ref_l = oracle.fork_decode_attn(b, rows=rows)
    out, lse = run_attn(b, flags=F8)
    assert np.isfinite(out).all()
    check_attn(out[rows[:, 0], rows[:, 1]], ref, lse[rows[:, 0], rows[:, 1]], ref_l, what="fp8 scores p128k",
               lse_max=LSE_FULL_SIZE_MAX_ABS)


@pytest.mark.parametrize("name,nrows", [("fp8_p128k_f32", 256), ("trace_p32k_f16", None)])
def test_peaked(name, nrows):
    b = synth.workload(name, kv_dtype="fp8_e4m3")
    rows = None if nrows is None else sample_rows(b, nrows, seed=12)
    peaked_check(b, "mfma", rows, f"fp8 scores peaked {name}", flags=F8)


def test_peaked_mid_size_all_rows():
    b = synth.make_fork_batch(prefix_lens=[3000, 900], forks_per_trace=[5, 2], suffix_range=(0, 300), num_q_heads=32,
                              num_kv_heads=4, head_dim=128, kv_dtype="fp8_e4m3", seed=410)
    peaked_check(b, "auto", None, "fp8 scores peaked mid", flags=F8)


@pytest.mark.parametrize("flags", [0, F8])
@pytest.mark.parametrize("path", ["auto", "mfma", "dot"])
def test_zero_scale_blocks(path, flags):
    """Blocks whose K or V scale is 0 (all-zero blocks quantise to scale 0):
    their values are 0 and their keys score 0, yet those keys still take part
    in the softmax.  Some prefix and suffix blocks get a zero V scale, some a
    zero K scale, one both; all rows against the oracle.  On the dot path the
    flag changes nothing: the same bits as without it."""
    b = synth.make_fork_batch(prefix_lens=[700], forks_per_trace=8, suffix_lens=[0, 5, 16, 40, 90, 1, 33, 64],
                              num_q_heads=32, num_kv_heads=4, head_dim=128, kv_dtype="fp8_e4m3", seed=470)
    pre = b.prefix_table[b.prefix_table_off[0]:b.prefix_table_off[0] + (700 + 15) // 16]
    suf = np.concatenate([b.suffix_table[b.suffix_table_off[f]:b.suffix_table_off[f] + (int(b.suffix_len[f]) + 15) // 16]
                          for f in range(b.num_forks)])
    b.v_scale[pre[[0, 5, 6, 43]]] = 0.0
    b.k_scale[pre[[2, 6, 20]]] = 0.0
    b.v_scale[suf[[1, 4]]] = 0.0
    b.k_scale[suf[[3]]] = 0.0
    ref, ref_l = oracle.fork_decode_attn(b)
    assert np.isfinite(ref).all() and np.isfinite(ref_l).all()
    say(f"zero scales: path {path} flags {flags}")
    o, l = run_attn(b, path, flags=flags)
    check_attn(o, ref, l, ref_l, what=f"zero-scale blocks, {path}, flags {flags}")
    if path == "dot" and flags:
        o0, l0 = run_attn(b, path)
        np.testing.assert_array_equal(o, o0)
        np.testing.assert_array_equal(l, l0)
