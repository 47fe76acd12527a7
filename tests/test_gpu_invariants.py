"""Properties of the HIP path that hold exactly: determinism, independence of
physical block placement, fork independence, no dependence on workspace
contents, and no state shared by calls in flight together on two streams."""
import copy

import numpy as np
import pytest
import torch

import paper_2606_17518_amd as sg
import synth
from gpu_helpers import run_attn, say

pytestmark = pytest.mark.gpu


def _batch(seed=5):
    return synth.make_fork_batch(prefix_lens=[700, 130], forks_per_trace=[6, 3], suffix_lens=[0, 5, 64, 65, 200, 17, 1, 33, 90],
                                 num_q_heads=32, num_kv_heads=4, head_dim=128, seed=seed)


@pytest.mark.parametrize("path", ["auto", "dot"])
def test_bitwise_deterministic(path):
    say(f"determinism {path}")
    b = _batch()
    o1, l1 = run_attn(b, path)
    o2, l2 = run_attn(b, path)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


def test_physical_placement_does_not_change_bits():
    say("paging invariance")
    b = _batch()
    rng = np.random.default_rng(11)
    perm = rng.permutation(b.num_blocks)          # block x moves to perm[x]
    c = copy.deepcopy(b)
    c.k_pool = np.empty_like(b.k_pool)
    c.v_pool = np.empty_like(b.v_pool)
    c.k_pool[perm] = b.k_pool
    c.v_pool[perm] = b.v_pool
    c.prefix_table = perm[b.prefix_table].astype(np.int32)
    c.suffix_table = perm[b.suffix_table].astype(np.int32)
    o1, l1 = run_attn(b)
    o2, l2 = run_attn(c)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


def test_fork_independence():
    say("fork independence")
    b = _batch()
    o1, l1 = run_attn(b)
    c = copy.deepcopy(b)
    f = 4
    ids = c.suffix_table[c.suffix_table_off[f]:c.suffix_table_off[f + 1]]
    c.v_pool[ids] = synth.fork_batch._to_bf16_bits(
        np.random.default_rng(3).standard_normal(c.v_pool[ids].shape).astype(np.float32))
    o2, l2 = run_attn(c)
    for g in range(b.num_forks):
        if g == f:
            assert not np.array_equal(o1[g], o2[g])
        else:
            assert np.array_equal(o1[g], o2[g]) and np.array_equal(l1[g], l2[g])


def test_workspace_contents_do_not_matter():
    say("workspace contents")
    b = _batch()
    fb = sg.ForkBatchTensors.from_numpy(b, "cuda")
    outs = []
    for fill in (0.0, float("nan"), 1e30):
        out = torch.empty((b.num_forks, b.num_q_heads, b.head_dim), dtype=torch.bfloat16, device="cuda")
        ws = sg.alloc_workspace(fb)
        ws.fill_(fill)
        sg.specgen_fork_decode_attn(fb, out, None, ws)
        torch.cuda.synchronize()
        outs.append(out.cpu())
    assert torch.equal(outs[0], outs[1]) and torch.equal(outs[0], outs[2])


def test_two_phases_equal_one_call():
    say("phases")
    b = _batch()
    fb = sg.ForkBatchTensors.from_numpy(b, "cuda")
    ws = sg.alloc_workspace(fb)
    o1 = torch.empty((b.num_forks, b.num_q_heads, b.head_dim), dtype=torch.bfloat16, device="cuda")
    l1 = torch.empty((b.num_forks, b.num_q_heads), dtype=torch.float32, device="cuda")
    o2, l2 = torch.empty_like(o1), torch.empty_like(l1)
    sg.specgen_fork_decode_attn(fb, o1, l1, ws)
    sg.specgen_fork_decode_attn_phase(fb, sg.SPECGEN_PHASE_PARTIALS, None, None, ws)
    sg.specgen_fork_decode_attn_phase(fb, sg.SPECGEN_PHASE_MERGE, o2, l2, ws)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_two_streams_at_once_give_the_serial_bits():
    """Two calls with their own workspaces and outputs in flight together on
    two streams (default priority) give the bits each gives alone: the calls
    share no device state."""
    say("two streams")
    b1 = synth.make_fork_batch(prefix_lens=[3000], forks_per_trace=6, suffix_range=(0, 300), num_q_heads=32,
                               num_kv_heads=4, head_dim=128, key_bias_std=0.5, seed=810)
    b2 = synth.make_fork_batch(prefix_lens=[900, 2000], forks_per_trace=[3, 5], suffix_range=(0, 200), num_q_heads=16,
                               num_kv_heads=2, head_dim=64, kv_dtype="fp8_e4m3", seed=811)
    batches = [(b, sg.ForkBatchTensors.from_numpy(b, "cuda")) for b in (b1, b2)]

    def buffers(b, fb):
        out = torch.full((b.num_forks, b.num_q_heads, b.head_dim), float("nan"), dtype=torch.bfloat16, device="cuda")
        lse = torch.full((b.num_forks, b.num_q_heads), float("nan"), dtype=torch.float32, device="cuda")
        return out, lse, sg.alloc_workspace(fb)

    alone = []
    for b, fb in batches:
        out, lse, ws = buffers(b, fb)
        sg.specgen_fork_decode_attn(fb, out, lse, ws)
        torch.cuda.synchronize()
        alone.append((out.clone(), lse.clone()))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    bufs = [buffers(b, fb) for b, fb in batches]
    torch.cuda.synchronize()
    for rep in range(5):
        for (b, fb), (out, lse, ws), st in zip(batches, bufs, streams):
            out.fill_(float("nan"))
            lse.fill_(float("nan"))
        torch.cuda.synchronize()
        for (b, fb), (out, lse, ws), st in zip(batches, bufs, streams):
            sg.specgen_fork_decode_attn(fb, out, lse, ws, stream=st)
        torch.cuda.synchronize()
        for (out, lse, _), (ao, al) in zip(bufs, alone):
            assert torch.equal(out.view(torch.int16), ao.view(torch.int16)), f"repeat {rep}"
            assert torch.equal(lse.view(torch.int32), al.view(torch.int32)), f"repeat {rep}"
