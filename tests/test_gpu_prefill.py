"""Multi-token fork prefill on the GPU (each fork's last q_len suffix tokens
are queries, causal inside the suffix), against the fp64 oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_17518_amd as sg
import synth
from gpu_helpers import check_attn, say

pytestmark = pytest.mark.gpu


def run_prefill(p, path="auto"):
    fb = sg.ForkBatchTensors.from_numpy(p, "cuda", path)
    Q, Hq, D = int(p.q_len.sum()), p.num_q_heads, p.head_dim
    out = torch.full((Q, Hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    lse = torch.full((Q, Hq), float("nan"), dtype=torch.float32, device="cuda")
    ws = sg.alloc_prefill_workspace(fb, p.q_len)
    ws.fill_(float("nan"))
    sg.specgen_fork_prefill_attn(fb, p.q_len, out, lse, ws)
    torch.cuda.synchronize()
    return out.float().cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)


CASES = {
    # one trace, ragged query counts, a query block that is the whole suffix
    "single": dict(batch=dict(prefix_lens=[300], forks_per_trace=4, suffix_lens=[5, 16, 40, 1], num_q_heads=16,
                              num_kv_heads=2, head_dim=128), q_len=[5, 3, 17, 1]),
    # nested prefixes with prefill
    "chain": dict(batch=dict(prefix_lens=[100, 33], prefix_parent=[-1, 0], forks_per_trace=[2, 2],
                             suffix_lens=[20, 8, 64, 2], num_q_heads=8, num_kv_heads=1, head_dim=64),
                  q_len=[4, 8, 30, 2]),
    # every fork has whole suffix blocks before its first query: they become a
    # nested prefix shared by the fork's queries (a trace with no forks of its own)
    "nest_single": dict(batch=dict(prefix_lens=[300], forks_per_trace=4, suffix_lens=[40, 21, 100, 33],
                                   num_q_heads=8, num_kv_heads=2, head_dim=64), q_len=[5, 5, 17, 1]),
    # one trace nests its forks' blocks, the trace below it cannot (a fork with 3 suffix tokens)
    "nest_mixed": dict(batch=dict(prefix_lens=[100, 50], prefix_parent=[-1, 0], forks_per_trace=[2, 2],
                                  suffix_lens=[40, 70, 3, 64], num_q_heads=16, num_kv_heads=2, head_dim=128),
                       q_len=[3, 10, 2, 20]),
    # many queries: 16 forks x 16 queries over an 8-head GQA group (2048 rows per kv head)
    "gqa8_q16": dict(batch=dict(prefix_lens=[1500], forks_per_trace=16, suffix_range=(16, 100), num_q_heads=64,
                                num_kv_heads=8, head_dim=128), q_len=[16] * 16),
    # the most queries one call takes: 4 traces x 8 forks x 16 queries = 512; forks
    # with 32 or more suffix tokens have a whole block before their first query,
    # so some traces nest their forks' blocks and others cannot
    "most_queries": dict(batch=dict(prefix_lens=[200, 90, 400, 33], forks_per_trace=8, suffix_range=(16, 80),
                                    num_q_heads=8, num_kv_heads=2, head_dim=64), q_len=[16] * 32),
}


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
@pytest.mark.parametrize("path", ["auto", "dot", "mfma"])
@pytest.mark.parametrize("name", list(CASES))
def test_prefill_matches_oracle(name, path, kv):
    say(f"prefill {name} path={path} kv={kv}")
    c = CASES[name]
    b = synth.make_fork_batch(kv_dtype=kv, seed=70 + list(CASES).index(name), **c["batch"])
    p = synth.with_prefill_queries(b, c["q_len"], seed=1)
    o, l = run_prefill(p, path)
    ro, rl = oracle.fork_prefill_attn(p, p.q_len)
    check_attn(o, ro, l, rl, what=f"prefill {name} {path} {kv}")


def test_prefill_of_one_query_equals_decode():
    say("prefill q_len=1 vs decode")
    b = synth.make_fork_batch(prefix_lens=[200], forks_per_trace=3, suffix_lens=[1, 17, 33], num_q_heads=16,
                              num_kv_heads=2, head_dim=128, seed=74)
    p = synth.with_prefill_queries(b, [1, 1, 1], seed=2)
    o, l = run_prefill(p)
    from gpu_helpers import run_attn
    b.q = p.q
    od, ld = run_attn(b)
    np.testing.assert_array_equal(o, od)
    np.testing.assert_array_equal(l, ld)


def test_prefill_full_size_sampled():
    """The 32768-token trace with 16 forks, each prefilling its last 16
    suffix tokens (256 queries x 64 q heads), on 48 sampled rows."""
    say("prefill full size trace_p32k_f16 q16")
    b = synth.workload("trace_p32k_f16")
    p = synth.with_prefill_queries(b, [16] * b.num_forks, seed=3)
    o, l = run_prefill(p)
    rng = np.random.default_rng(4)
    Q = int(p.q_len.sum())
    idx = np.unique(np.concatenate([[0, Q * p.num_q_heads - 1], rng.choice(Q * p.num_q_heads, 46, replace=False)]))
    rows = np.stack([idx // p.num_q_heads, idx % p.num_q_heads], axis=1).astype(np.int32)
    ro, rl = oracle.fork_prefill_attn(p, p.q_len, rows=rows)
    check_attn(o[rows[:, 0], rows[:, 1]], ro, l[rows[:, 0], rows[:, 1]], rl, what="prefill full size")
