"""The no-allocation entry point (specgen_fork_decode_attn_noalloc) against the
workspace entry point (specgen_fork_decode_attn) on the GPU, through the C ABI.

Two calls in a row share the library's per-GPU scratch: first the 32k-prefix
16-fork decode step (about 50 MB of partials), then the tiny 256-token batch.
Each must give exactly the bits the workspace call gives for the same batch
(same plan, same kernels, no floating-point atomics), and the tiny one also
matches the fp64 oracle within the attention tolerances.  A batch whose
workspace exceeds the scratch is rejected before anything is queued.
"""
import ctypes as C

import numpy as np
import pytest
import torch

import oracle
import paper_2606_17518_amd as sg
import synth
from gpu_helpers import check_attn, say

pytestmark = pytest.mark.gpu


def _outputs(fb, N, Hq, D):
    out = torch.full((N, Hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    lse = torch.full((N, Hq), float("nan"), dtype=torch.float32, device="cuda")
    return out, lse


def _noalloc(fb, out, lse):
    s = fb.c_struct()
    st = sg.lib().specgen_fork_decode_attn_noalloc(C.byref(s), C.c_void_p(out.data_ptr()),
                                                   C.c_void_p(lse.data_ptr()),
                                                   C.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == sg.binding.SPECGEN_OK, sg.lib().specgen_last_error().decode()


def test_noalloc_matches_the_workspace_call_twice_in_a_row():
    results = []
    for name in ("trace_p32k_f16", "tiny_p256_f4"):   # the second call is the smaller one
        say(f"noalloc: {name}: generating")
        b = synth.workload(name)
        fb = sg.ForkBatchTensors.from_numpy(b, "cuda")
        N, Hq, D = b.num_forks, b.num_q_heads, b.head_dim
        assert sg.specgen_fork_decode_attn_workspace_size(fb) <= sg.SPECGEN_NOALLOC_SCRATCH_BYTES
        out_n, lse_n = _outputs(fb, N, Hq, D)
        say(f"noalloc: {name}: no-allocation call")
        _noalloc(fb, out_n, lse_n)
        torch.cuda.synchronize()
        say(f"noalloc: {name}: workspace call")
        out_w, lse_w = _outputs(fb, N, Hq, D)
        ws = sg.alloc_workspace(fb)
        ws.fill_(float("nan"))
        sg.specgen_fork_decode_attn(fb, out_w, lse_w, ws)
        torch.cuda.synchronize()
        assert torch.equal(out_n.view(torch.int16), out_w.view(torch.int16)), f"{name}: output bits differ"
        assert torch.equal(lse_n.view(torch.int32), lse_w.view(torch.int32)), f"{name}: lse bits differ"
        results.append((b, out_n, lse_n))
        del ws, fb
    b, out_n, lse_n = results[1]
    ref, ref_l = oracle.fork_decode_attn(b)
    check_attn(out_n.float().cpu().numpy().astype(np.float64), ref, lse_n.cpu().numpy().astype(np.float64), ref_l,
               what="noalloc tiny vs oracle")
    # the first (larger) call's output is still what it was: nothing wrote into it
    assert torch.isfinite(results[0][1].float()).all()


def test_noalloc_rejects_a_batch_above_the_scratch():
    b = synth.make_fork_batch(prefix_lens=[131072], forks_per_trace=32, suffix_lens=[16] * 32, num_q_heads=128,
                              num_kv_heads=8, head_dim=128, kv_dtype="fp8_e4m3", extra_blocks=0, seed=4)
    fb = sg.ForkBatchTensors.from_numpy(b, "cuda")
    assert sg.specgen_fork_decode_attn_workspace_size(fb) > sg.SPECGEN_NOALLOC_SCRATCH_BYTES
    out, lse = _outputs(fb, b.num_forks, b.num_q_heads, b.head_dim)
    s = fb.c_struct()
    st = sg.lib().specgen_fork_decode_attn_noalloc(C.byref(s), C.c_void_p(out.data_ptr()), C.c_void_p(lse.data_ptr()),
                                                   None)
    assert st == sg.binding.SPECGEN_ERR_WORKSPACE
    assert "scratch" in sg.lib().specgen_last_error().decode()
    torch.cuda.synchronize()
    assert torch.isnan(out.float()).all(), "a rejected call wrote its output"
