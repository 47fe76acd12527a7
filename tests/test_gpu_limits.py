"""Batches at the boundary's per-call limits on the GPU, every row against the
oracle:
  - 32 traces with 16 forks each, 512 forks in all (the most one call takes),
    prefixes of 1-300 tokens and suffixes of 0-60 (a fifth empty), so each
    worker's range crosses many small items of both kinds;
  - the largest GQA group, 128 query heads on one kv head: a trace of 3 forks
    has 384 rows per kv head (items of 256 and 128 rows), one of 2 forks 256.
Both KV dtypes and all three kernel paths.  Rows whose fork sees fewer than 32
keys are about one value row, so the bar there is the error beyond the bf16
output's own rounding; elsewhere the attention tolerances.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import check_attn, check_attn_excess, run_attn, say

pytestmark = pytest.mark.gpu


def _check_all_rows(b, path, what):
    ref, ref_l = oracle.fork_decode_attn(b)
    out, lse = run_attn(b, path)
    keys = np.array([b.keys_of_fork(f) for f in range(b.num_forks)])
    few = keys < 32
    if few.any():
        check_attn_excess(out[few], ref[few], lse[few], ref_l[few], what=f"{what}, forks of < 32 keys")
    if (~few).any():
        check_attn(out[~few], ref[~few], lse[~few], ref_l[~few], what=what)


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
@pytest.mark.parametrize("path", ["auto", "mfma", "dot"])
def test_most_traces_and_forks_per_call(path, kv):
    rng = np.random.default_rng(7100)
    T, F = 32, 16
    P = [int(x) for x in rng.integers(1, 301, size=T)]
    S = [0 if rng.random() < 0.2 else int(x) for x in rng.integers(1, 61, size=T * F)]
    b = synth.make_fork_batch(prefix_lens=P, forks_per_trace=F, suffix_lens=S, num_q_heads=8, num_kv_heads=2,
                              head_dim=64, kv_dtype=kv, key_bias_std=0.5, seed=7101)
    assert b.num_traces == 32 and b.num_forks == 512
    say(f"limits: 32 traces x 16 forks, {kv}, path={path}")
    _check_all_rows(b, path, f"512 forks {kv} {path}")


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
@pytest.mark.parametrize("path", ["auto", "mfma", "dot"])
def test_largest_gqa_group(path, kv):
    b = synth.make_fork_batch(prefix_lens=[700, 333], forks_per_trace=[3, 2], suffix_lens=[0, 45, 130, 17, 1],
                              num_q_heads=128, num_kv_heads=1, head_dim=128, kv_dtype=kv, key_bias_std=0.5,
                              seed=7102)
    say(f"limits: GQA group 128, {kv}, path={path}")
    _check_all_rows(b, path, f"group 128 {kv} {path}")
