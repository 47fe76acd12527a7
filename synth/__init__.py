"""Seeded synthetic workloads shared by the oracle and the HIP path.

The five named workloads stand in for the KV caches of long reasoning traces
with speculative forks (Sec. 4.2 puts useful fork points at 14-70% of a trace;
Table "tab:token_overhead" implies roughly 24k tokens per iteration).  The
paper's own workloads (LLM reasoning traces over KernelBench tasks) are not
reproduced; these synthetic tensors have the shapes of such caches.
"""
from .fork_batch import (BLOCK, AppendCase, ForkBatch, ImportCase, make_append_case, make_fork_batch,
                         make_import_case, prefix_import_from_batch, SENTINEL, with_prefill_queries)

# name -> (fork-batch keyword arguments, import description or None)
WORKLOADS = {
    # 1 prefix of 256 tokens, 4 forks with suffixes in [0, 32], GQA 8/2, D=64,
    # shuffled 64-block pool; import of the 16 prefix blocks
    "tiny_p256_f4": dict(
        batch=dict(prefix_lens=[256], forks_per_trace=4, suffix_range=(0, 32), num_q_heads=8,
                   num_kv_heads=2, head_dim=64, num_blocks=64),
        import_prefix=True),
    # single trace: P=8192, 8 forks with suffixes in [64, 512], GQA 64/8, D=128
    "trace_p8k_f8": dict(
        batch=dict(prefix_lens=[8192], forks_per_trace=8, suffix_range=(64, 512), num_q_heads=64,
                   num_kv_heads=8, head_dim=128),
        import_prefix=False),
    # long trace, heavy forking: P=32768, 16 forks, suffixes in [128, 1024],
    # keys with a per-kv-head bias of std 0.5, 16384-block pool; import of the
    # 2048 prefix blocks through the random permutation table
    "trace_p32k_f16": dict(
        batch=dict(prefix_lens=[32768], forks_per_trace=16, suffix_range=(128, 1024), num_q_heads=64,
                   num_kv_heads=8, head_dim=128, key_bias_std=0.5, num_blocks=16384),
        import_prefix=True),
    # ragged: 32 traces, P in [4096, 32768], 8 forks each, suffixes in [0, 2048]
    "ragged_t32_f8": dict(
        batch=dict(prefix_range=(4096, 32768), num_traces=32, forks_per_trace=8, suffix_range=(0, 2048),
                   num_q_heads=64, num_kv_heads=8, head_dim=128, extra_blocks=0),
        import_prefix=False),
    # extreme prefix with E4M3 KV: P=131072, 32 forks, suffixes in [256, 4096], GQA 128/8
    "fp8_p128k_f32": dict(
        batch=dict(prefix_lens=[131072], forks_per_trace=32, suffix_range=(256, 4096), num_q_heads=128,
                   num_kv_heads=8, head_dim=128, kv_dtype="fp8_e4m3", extra_blocks=0),
        import_prefix=False),
    # nested fork points on one 32768-token trace (a fork tree): forks taken at
    # 16384 tokens (4), at 24576 (6) and at 32768 (6) see prefixes that extend
    # each other, stored once as three segments of 16384, 8192 and 8192 tokens;
    # suffixes in [128, 1024], keys with the per-kv-head bias of std 0.5
    "tree_p32k_l3": dict(
        batch=dict(prefix_lens=[16384, 8192, 8192], prefix_parent=[-1, 0, 1], forks_per_trace=[4, 6, 6],
                   suffix_range=(128, 1024), num_q_heads=64, num_kv_heads=8, head_dim=128, key_bias_std=0.5,
                   num_blocks=16384),
        import_prefix=False),
    # multi-token prefill over the P=32768 trace of trace_p32k_f16: each of its
    # 16 forks processes its last 16 suffix tokens as queries (256 queries)
    "prefill_p32k_f16_q16": dict(
        batch=dict(prefix_lens=[32768], forks_per_trace=16, suffix_range=(128, 1024), num_q_heads=64,
                   num_kv_heads=8, head_dim=128, key_bias_std=0.5, num_blocks=16384),
        import_prefix=False, prefill_q=16),
}
WORKLOAD_SEEDS = {name: i + 1 for i, name in enumerate(WORKLOADS)}


def workload(name: str, seed: int | None = None, **overrides) -> ForkBatch:
    spec = dict(WORKLOADS[name]["batch"])
    spec.update(overrides)
    return make_fork_batch(seed=WORKLOAD_SEEDS[name] if seed is None else seed, name=name, **spec)
