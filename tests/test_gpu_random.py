"""Randomised parity sweep of fork-decode attention on the GPU against the fp64
oracle, all rows of every case.

Each case draws (from its own seed) a fork tree of 1-4 traces (nested
prefixes in depth-first order, or independent roots), 1-4 forks per trace,
prefix lengths 1-600, suffix lengths 0-300 (a fifth of the forks without a
suffix; a wide set: 2-8 forks per trace, prefixes of 1000-6000, suffixes up to
1000), GQA group size 1-16 over 1-8 kv heads, head_dim 64 or 128, bf16 or
E4M3 KV, a per-head key bias or none, the kernel path (auto, MFMA or dot) and,
for E4M3 at head_dim 128 off the dot path, fp8 scores half the time.  The
shapes land on every work-split and merge variant: one or several items per
workgroup, one or two token groups, the grouped and the one-row-per-wave
merges.  Rows whose fork sees fewer than 32 keys are about one value row, so
the bar there is the error beyond the bf16 output's own rounding; elsewhere the
plain tolerances.
"""
import numpy as np
import pytest

import oracle
import paper_2606_17518_amd as sg
import synth
from gpu_helpers import check_attn, check_attn_excess, run_attn, say

pytestmark = pytest.mark.gpu
CASES = 96
WIDE = 24   # longer prefixes and suffixes, more forks: items over several workgroups, rows of many parts


def _case(i, wide=False):
    rng = np.random.default_rng(9000 + i + (5000 if wide else 0))
    T = int(rng.integers(1, 5))
    parent = [-1]
    for t in range(1, T):
        choices = [-1, t - 1]   # a root, the previous trace or one of its ancestors (depth-first order)
        a = parent[t - 1]
        while a >= 0:
            choices.append(a)
            a = parent[a]
        parent.append(int(rng.choice(choices)))
    F = [int(x) for x in rng.integers(2 if wide else 1, 9 if wide else 5, size=T)]
    N = sum(F)
    P = [int(x) for x in rng.integers(1000 if wide else 1, 6001 if wide else 601, size=T)]
    S = [0 if rng.random() < 0.2 else int(x) for x in rng.integers(1, 1001 if wide else 301, size=N)]
    Hkv = int(rng.choice([1, 2, 4, 8]))
    g = int(rng.choice([1, 2, 4, 8, 16]))
    D = int(rng.choice([64, 128]))
    kv = "fp8_e4m3" if rng.random() < 0.35 else "bf16"
    path = str(rng.choice(["auto", "mfma", "dot"]))
    flags = sg.SPECGEN_FLAG_FP8_SCORES if (kv != "bf16" and D == 128 and path != "dot" and rng.random() < 0.5) else 0
    bias = float(rng.choice([0.0, 0.5]))
    nested = any(p >= 0 for p in parent)
    b = synth.make_fork_batch(prefix_lens=P, forks_per_trace=F, suffix_lens=S, num_q_heads=g * Hkv,
                              num_kv_heads=Hkv, head_dim=D, kv_dtype=kv, key_bias_std=bias,
                              seed=9100 + i + (5000 if wide else 0),
                              prefix_parent=parent if nested else None)
    desc = (f"T={T} parent={parent} F={F} P={P} S={S} Hkv={Hkv} g={g} D={D} {kv} path={path} flags={flags} "
            f"bias={bias}")
    return b, path, flags, desc


@pytest.mark.parametrize("i,wide", [(i, False) for i in range(CASES)] + [(i, True) for i in range(WIDE)])
def test_random_case_all_rows(i, wide):
    b, path, flags, desc = _case(i, wide)
    say(f"random case {i}: {desc}")
    ref, ref_l = oracle.fork_decode_attn(b)
    out, lse = run_attn(b, path, flags=flags)
    keys = np.array([b.keys_of_fork(f) for f in range(b.num_forks)])
    few = keys < 32
    if few.any():
        check_attn_excess(out[few], ref[few], lse[few], ref_l[few], what=f"random {i}, forks of < 32 keys")
    if (~few).any():
        check_attn(out[~few], ref[~few], lse[~few], ref_l[~few], what=f"random {i}")
