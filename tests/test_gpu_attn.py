"""Fork-decode attention on the GPU against the fp64 oracle.

Tolerance (bf16 inputs, fp32 accumulation, bf16 output): max abs <= 1e-2 and
mean abs <= 1e-3 over all compared elements; natural-log LSE within 1e-3.
Small shapes and the 32k-prefix workload are compared on every row; the other
long workloads on sampled rows (the oracle computes each sampled row by
definition over its full key set).  The full-size workloads also meet an lse
bound of 1e-4, which a single dropped 16-token block would break.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import LSE_FULL_SIZE_MAX_ABS, check_attn, run_attn, sample_rows, say

pytestmark = pytest.mark.gpu

# (prefix lens, forks per trace, suffix lens, Hq, Hkv, D, kv dtype)
SMALL = [
    ([1], 1, [0], 8, 8, 64, "bf16"),                    # one key, MHA
    ([15], 2, [1, 0], 8, 2, 128, "bf16"),
    ([16], 3, [15, 16, 17], 16, 2, 128, "bf16"),        # r = 24
    ([17], 4, [0, 1, 15, 16], 4, 4, 64, "bf16"),        # g = 1, r = 4
    ([100], 8, [0, 1, 15, 16, 17, 31, 32, 33], 16, 1, 128, "bf16"),  # g = 16, r = 128
    ([129], 2, [64, 65], 32, 2, 64, "bf16"),            # r = 32
    ([1000], 5, [7, 300, 0, 64, 129], 64, 8, 128, "bf16"),  # r = 40
    ([777], 16, list(range(0, 160, 10)), 64, 8, 128, "bf16"),  # r = 128, ragged tail
    ([2048], 9, [5] * 9, 72, 4, 128, "bf16"),           # r = 162: two row blocks
    ([3, 70, 16], [1, 3, 2], [2, 0, 40, 17, 1, 16], 8, 2, 64, "bf16"),  # three traces
    ([300], 4, [0, 3, 33, 70], 16, 2, 128, "fp8_e4m3"),
    ([65, 190], [2, 3], [1, 0, 16, 17, 80], 32, 8, 64, "fp8_e4m3"),
    # items of more than 128 rows: two q slots, one token group per wave
    ([300], 16, list(range(0, 320, 20)), 256, 16, 128, "bf16"),      # r = 256: 8 row groups
    ([200], 12, [3, 64, 65, 0, 7, 128, 1, 33, 90, 2, 15, 16], 240, 16, 64, "bf16"),  # r = 180, D = 64
    ([500], 16, list(range(5, 165, 10)), 256, 16, 128, "fp8_e4m3"),  # r = 256 with E4M3
    ([130], 20, [1] * 20, 160, 8, 64, "fp8_e4m3"),                   # r = 400: row blocks of 256 and 144
]


def _small(i):
    P, F, S, Hq, Hkv, D, dt = SMALL[i]
    return synth.make_fork_batch(prefix_lens=P, forks_per_trace=F, suffix_lens=S, num_q_heads=Hq,
                                 num_kv_heads=Hkv, head_dim=D, kv_dtype=dt, seed=100 + i)


@pytest.mark.parametrize("path", ["auto", "mfma", "dot"])
@pytest.mark.parametrize("i", range(len(SMALL)))
def test_small_shapes_all_rows(i, path):
    b = _small(i)
    say(f"small case {i} {SMALL[i]} path={path}")
    ref, ref_l = oracle.fork_decode_attn(b)
    out, lse = run_attn(b, path)
    check_attn(out, ref, lse, ref_l, what=f"case {i} {path}")


@pytest.mark.parametrize("path", ["auto", "mfma", "dot"])
def test_tiny_workload_all_rows(path):
    b = synth.workload("tiny_p256_f4")
    say(f"tiny_p256_f4 path={path}")
    ref, ref_l = oracle.fork_decode_attn(b)
    out, lse = run_attn(b, path)
    check_attn(out, ref, lse, ref_l, what="tiny")


def test_trace_8k_all_rows():
    b = synth.workload("trace_p8k_f8")
    say("trace_p8k_f8 all rows")
    ref, ref_l = oracle.fork_decode_attn(b)
    out, lse = run_attn(b)
    check_attn(out, ref, lse, ref_l, what="p8k")


@pytest.mark.parametrize("name,nrows", [("trace_p32k_f16", None), ("ragged_t32_f8", 1024), ("fp8_p128k_f32", 256)])
def test_full_size_workloads(name, nrows):
    """Full-size decode workloads: every row of the 32k-prefix workload, sampled
    rows of the others (the oracle computes each by definition over all its
    keys); the attention tolerances, and beside them the lse bound that
    resolves a single 16-token block."""
    say(f"{name}: generating")
    b = synth.workload(name)
    rows = None if nrows is None else sample_rows(b, nrows, seed=7)
    say(f"{name}: oracle on {'all' if rows is None else len(rows)} rows")
    ref, ref_l = oracle.fork_decode_attn(b, rows=rows)
    say(f"{name}: gpu")
    out, lse = run_attn(b)
    assert np.isfinite(out).all()
    if rows is None:
        got, got_l = out, lse
    else:
        got, got_l = out[rows[:, 0], rows[:, 1]], lse[rows[:, 0], rows[:, 1]]
    check_attn(got, ref, got_l, ref_l, what=name, lse_max=LSE_FULL_SIZE_MAX_ABS)
