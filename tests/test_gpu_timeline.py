"""The timeline build (libspecgen_timeline.so, SPECGEN_TIMELINE) on the GPU:
its partial kernel gives the release library's bits, and every workgroup that
ran leaves ordered stamps (start <= plan copied <= walk done <= each slot
landed <= end) and its slot count."""
import ctypes as C

import numpy as np
import pytest
import torch

import paper_2606_17518_amd as sg
import synth
from gpu_helpers import say

pytestmark = pytest.mark.gpu
B = sg.binding


def _call(L, fb, out, lse, ws):
    return L.specgen_fork_decode_attn(C.byref(fb.c_struct()), C.c_void_p(out.data_ptr()), C.c_void_p(lse.data_ptr()),
                                      C.c_void_p(ws.data_ptr()), ws.numel() * 4,
                                      C.c_void_p(torch.cuda.current_stream().cuda_stream))


@pytest.mark.parametrize("name", ["tiny_p256_f4", "trace_p8k_f8"])
def test_timeline_build_bits_and_stamps(name):
    b = synth.workload(name)
    fb = sg.ForkBatchTensors.from_numpy(b, "cuda")
    ws = sg.alloc_workspace(fb)
    T = B.timeline_lib()
    res = []
    for L, tag in ((sg.lib(), "release"), (T, "timeline")):
        say(f"timeline: {name}, {tag} library")
        out = torch.empty((b.num_forks, b.num_q_heads, b.head_dim), dtype=torch.bfloat16, device="cuda")
        lse = torch.empty((b.num_forks, b.num_q_heads), dtype=torch.float32, device="cuda")
        if L is T:
            assert T.specgen_timeline_clear() == 0
        assert _call(L, fb, out, lse, ws) == B.SPECGEN_OK, L.specgen_last_error().decode()
        torch.cuda.synchronize()
        res.append((out, lse))
    assert torch.equal(res[0][0].view(torch.int16), res[1][0].view(torch.int16))
    assert torch.equal(res[0][1].view(torch.int32), res[1][1].view(torch.int32))
    W, S = C.c_int(0), C.c_int(0)
    assert T.specgen_timeline_shape(C.byref(W), C.byref(S)) == 0
    W, S = W.value, S.value
    st = np.zeros((W, S), np.uint64)
    kd = np.zeros((W, S), np.int32)
    assert T.specgen_timeline_read(st.ctypes.data, kd.ctypes.data) == 0
    live = np.nonzero(st[:, 0])[0]
    assert live.size > 0 and live.max() < W
    for w in live:
        n = int(kd[w, S - 1])
        assert n >= 0
        seq = [st[w, 0], st[w, 1], st[w, 2], st[w, 3]] + [st[w, 4 + s] for s in range(min(n, S - 5))] + [st[w, S - 1]]
        if n == 0:   # a worker with no tiles ends after its walk
            seq = [st[w, 0], st[w, 1], st[w, 2], st[w, S - 1]]
        assert all(x > 0 for x in seq), (w, seq)
        assert all(a <= c for a, c in zip(seq, seq[1:])), (w, seq)
        assert list(kd[w, :3]) == [100, 101, 102]
        if n > 0:
            assert kd[w, 3] == 103
        if n > 0:
            assert kd[w, 4] == -1   # every range starts with its first item's q slot
            assert set(kd[w, 4:4 + min(n, S - 5)]) <= {-1, 0, 1}
