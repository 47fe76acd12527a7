"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
and compare with the fp64 oracle to the stated tolerances."""
import sys

import numpy as np
import torch

import oracle
import paper_2606_17518_amd as sg

# attention tolerances on bf16 out vs the fp64 oracle (bf16 inputs, fp32 accumulation)
ATTN_MAX_ABS = 1e-2
ATTN_MEAN_ABS = 1e-3
LSE_MAX_ABS = 1e-3


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def run_attn(batch, path="auto", with_lse=True, fb=None):
    if fb is None:
        fb = sg.ForkBatchTensors.from_numpy(batch, "cuda", path)
    N, Hq, D = batch.num_forks, batch.num_q_heads, batch.head_dim
    out = torch.full((N, Hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    lse = torch.full((N, Hq), float("nan"), dtype=torch.float32, device="cuda") if with_lse else None
    ws = sg.alloc_workspace(fb)
    ws.fill_(float("nan"))
    sg.specgen_fork_decode_attn(fb, out, lse, ws)
    torch.cuda.synchronize()
    o = out.float().cpu().numpy().astype(np.float64)
    l = lse.cpu().numpy().astype(np.float64) if with_lse else None
    return o, l


def check_attn(out, ref, lse=None, ref_lse=None, what=""):
    assert np.isfinite(out).all(), f"{what}: non-finite output"
    err = np.abs(out - ref)
    mx, mean = float(err.max()), float(err.mean())
    assert mx <= ATTN_MAX_ABS, f"{what}: max abs err {mx:.3e}"
    assert mean <= ATTN_MEAN_ABS, f"{what}: mean abs err {mean:.3e}"
    if lse is not None:
        le = float(np.abs(lse - ref_lse).max())
        assert le <= LSE_MAX_ABS, f"{what}: lse max abs err {le:.3e}"
    return mx, mean


def sample_rows(batch, n, seed=0):
    """n distinct (fork, q head) rows, always including the first and last."""
    rng = np.random.default_rng(seed)
    total = batch.num_forks * batch.num_q_heads
    idx = np.unique(np.concatenate([[0, total - 1], rng.choice(total, size=min(n, total), replace=False)]))
    return np.stack([idx // batch.num_q_heads, idx % batch.num_q_heads], axis=1).astype(np.int32)
