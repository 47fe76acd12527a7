"""Fork-decode attention captured in a HIP graph (torch.cuda.CUDAGraph): the
call allocates nothing and records no memset, so a captured step replays
with whatever the input buffers hold at replay time.  Every replay is
checked against an eager call on the same inputs and against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_17518_amd as sg
import synth
from gpu_helpers import check_attn, say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,kw", [
    ("p256_f4", dict(prefix_lens=[256], forks_per_trace=4, suffix_range=(0, 32), num_q_heads=8, num_kv_heads=2,
                     head_dim=64)),
    ("p4k_f8_e4m3", dict(prefix_lens=[4000], forks_per_trace=8, suffix_range=(10, 300), num_q_heads=64,
                         num_kv_heads=8, head_dim=128, kv_dtype="fp8_e4m3")),
])
def test_graph_replays_match_eager(name, kw):
    say(f"graph {name}")
    b = synth.make_fork_batch(seed=90, **kw)
    fb = sg.ForkBatchTensors.from_numpy(b)
    N, Hq, D = b.num_forks, b.num_q_heads, b.head_dim
    out = torch.zeros((N, Hq, D), dtype=torch.bfloat16, device="cuda")
    lse = torch.zeros((N, Hq), dtype=torch.float32, device="cuda")
    ws = sg.alloc_workspace(fb)
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):   # warm the library and HIP module loads outside the capture
        sg.specgen_fork_decode_attn(fb, out, lse, ws, stream=stream)
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        sg.specgen_fork_decode_attn(fb, out, lse, ws, stream=stream)
    rng = np.random.default_rng(1)
    for rep in range(3):
        # new queries in the captured buffer, eager work in between
        q = synth.fork_batch._to_bf16_bits(rng.standard_normal((N, Hq, D), dtype=np.float32))
        fb.q.copy_(torch.from_numpy(q.view(np.int16)).cuda())
        out.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        o = out.float().cpu().numpy().astype(np.float64)
        l = lse.cpu().numpy().astype(np.float64)
        e_out = torch.empty_like(out)
        e_lse = torch.empty_like(lse)
        e_ws = sg.alloc_workspace(fb)
        sg.specgen_fork_decode_attn(fb, e_out, e_lse, e_ws)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(o, e_out.float().cpu().numpy().astype(np.float64))
        np.testing.assert_array_equal(l, e_lse.cpu().numpy().astype(np.float64))
        b.q = q
        ro, rl = oracle.fork_decode_attn(b)
        check_attn(o, ro, l, rl, what=f"graph replay {rep}")
