"""The debug build (libspecgen_debug.so, SPECGEN_DEBUG_CHECKS) on the GPU.

It runs the same kernels as the release library, so a valid batch gives the
same bits; and it checks every attention block id on the host before any
launch.  The "bad" ids used here are out of range only for the num_blocks the
call is given: they index blocks that exist in the pool tensors, so even a
launch would read allocated memory.  Every rejected call must leave its
outputs untouched.
"""
import ctypes as C

import numpy as np
import pytest
import torch

import paper_2606_17518_amd as sg
import synth
from gpu_helpers import say

pytestmark = pytest.mark.gpu
B = sg.binding


def _used_ids(b):
    """(table, owner, entry, id) of every id the attention reads, traces first."""
    out = []
    for t in range(b.num_traces):
        o, n = int(b.prefix_table_off[t]), (int(b.prefix_len[t]) + 15) // 16
        out += [("prefix", t, o + i, int(b.prefix_table[o + i])) for i in range(n)]
    for f in range(b.num_forks):
        o, n = int(b.suffix_table_off[f]), (int(b.suffix_len[f]) + 15) // 16
        out += [("suffix", f, o + i, int(b.suffix_table[o + i])) for i in range(n)]
    return out


def _bufs(b):
    out = torch.full((b.num_forks, b.num_q_heads, b.head_dim), float("nan"), dtype=torch.bfloat16, device="cuda")
    lse = torch.full((b.num_forks, b.num_q_heads), float("nan"), dtype=torch.float32, device="cuda")
    return out, lse


def _call(L, s, out, lse, ws):
    return L.specgen_fork_decode_attn(C.byref(s), C.c_void_p(out.data_ptr()), C.c_void_p(lse.data_ptr()),
                                      C.c_void_p(ws.data_ptr()), ws.numel() * 4,
                                      C.c_void_p(torch.cuda.current_stream().cuda_stream))


def _untouched(out, lse):
    torch.cuda.synchronize()
    return bool(torch.isnan(out.float()).all()) and bool(torch.isnan(lse).all())


@pytest.fixture(scope="module")
def tiny():
    b = synth.workload("tiny_p256_f4")
    return b, sg.ForkBatchTensors.from_numpy(b, "cuda")


def test_debug_build_gives_the_release_bits(tiny):
    b, fb = tiny
    D = B.debug_lib()
    ws = sg.alloc_workspace(fb)
    res = []
    for L, name in ((sg.lib(), "release"), (D, "debug")):
        say(f"debug checks: valid batch, {name} library")
        out, lse = _bufs(b)
        ws.fill_(float("nan"))
        st = _call(L, fb.c_struct(), out, lse, ws)
        assert st == B.SPECGEN_OK, L.specgen_last_error().decode()
        torch.cuda.synchronize()
        res.append((out, lse))
    assert torch.equal(res[0][0].view(torch.int16), res[1][0].view(torch.int16))
    assert torch.equal(res[0][1].view(torch.int32), res[1][1].view(torch.int32))


def test_debug_build_rejects_a_prefix_id_at_num_blocks(tiny):
    b, fb = tiny
    D = B.debug_lib()
    used = _used_ids(b)
    top = max(i for tb, _, _, i in used if tb == "prefix")
    first_bad = next(u for u in used if u[3] >= top)
    assert first_bad[0] == "prefix"
    s = fb.c_struct(num_blocks=top)   # ids == top are now out of range; the pool still holds them
    ws = sg.alloc_workspace(fb)
    out, lse = _bufs(b)
    say("debug checks: prefix id == num_blocks")
    st = _call(D, s, out, lse, ws)
    msg = D.specgen_last_error().decode()
    assert st == B.SPECGEN_ERR_INVALID_ARG, msg
    assert f"prefix_table[{first_bad[2]}] = {first_bad[3]}" in msg and f"trace {first_bad[1]}" in msg, msg
    assert _untouched(out, lse)
    # the other launching entry points reject it the same way
    st = D.specgen_fork_decode_attn_phase(C.byref(s), B.SPECGEN_PHASE_PARTIALS, None, None,
                                          C.c_void_p(ws.data_ptr()), ws.numel() * 4, None)
    assert st == B.SPECGEN_ERR_INVALID_ARG
    st = D.specgen_fork_decode_attn_noalloc(C.byref(s), C.c_void_p(out.data_ptr()), C.c_void_p(lse.data_ptr()), None)
    assert st == B.SPECGEN_ERR_INVALID_ARG
    q_len = np.ones(b.num_forks, np.int32)
    n = C.c_size_t(0)
    assert D.specgen_fork_prefill_attn_workspace_size(C.byref(s), q_len.ctypes.data, C.byref(n)) == B.SPECGEN_OK
    wsp = torch.empty(max(n.value, 256) // 4 + 64, dtype=torch.float32, device="cuda")
    st = D.specgen_fork_prefill_attn(C.byref(s), q_len.ctypes.data, C.c_void_p(out.data_ptr()),
                                     C.c_void_p(lse.data_ptr()), C.c_void_p(wsp.data_ptr()), wsp.numel() * 4, None)
    assert st == B.SPECGEN_ERR_INVALID_ARG
    assert _untouched(out, lse)


def test_debug_build_rejects_a_suffix_id_past_num_blocks(tiny):
    b, fb = tiny
    D = B.debug_lib()
    used = _used_ids(b)
    top = max(i for _, _, _, i in used)
    assert top + 1 < b.num_blocks   # block top + 1 exists in the pool
    # fork 2's second suffix block becomes top + 1, which is out of range for num_blocks = top + 1
    f = 2
    e = int(b.suffix_table_off[f]) + 1
    assert (int(b.suffix_len[f]) + 15) // 16 >= 2
    tab = fb.suffix_table.clone()
    tab[e] = top + 1
    s = fb.c_struct(num_blocks=top + 1, suffix_table=tab.data_ptr())
    ws = sg.alloc_workspace(fb)
    out, lse = _bufs(b)
    say("debug checks: suffix id past num_blocks")
    st = _call(D, s, out, lse, ws)
    msg = D.specgen_last_error().decode()
    assert st == B.SPECGEN_ERR_INVALID_ARG, msg
    assert f"suffix_table[{e}] = {top + 1}" in msg and f"fork {f}" in msg, msg
    assert _untouched(out, lse)
    # with the table restored the same claimed size is valid again
    s = fb.c_struct(num_blocks=top + 1)
    assert _call(D, s, out, lse, ws) == B.SPECGEN_OK, D.specgen_last_error().decode()
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all()
