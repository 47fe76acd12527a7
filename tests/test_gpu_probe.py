"""The benchmark's memory-ceiling probes (libspecgen_probe.so) on the GPU:
each queues its kernel, returns 0 and leaves the sink untouched on data whose
xor is not the sentinel.  The slice ring runs on a small pool, with more
workgroups than tiles (idle workgroups) and with ids outside the pool (the
probe clamps them)."""
import ctypes as C

import numpy as np
import pytest
import torch

from gpu_helpers import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    from paper_2606_17518_amd.build import PROBE_LIB_PATH
    lib = C.CDLL(PROBE_LIB_PATH)
    lib.specgen_probe_stream_read.argtypes = [C.c_void_p, C.c_int64, C.c_void_p, C.c_void_p]
    lib.specgen_probe_stream_copy.argtypes = [C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p]
    lib.specgen_probe_slice_ring.argtypes = [C.c_void_p, C.c_void_p, C.c_int64, C.c_int, C.c_void_p, C.c_int, C.c_int,
                                             C.c_void_p, C.c_void_p]
    return lib


def test_stream_copy_copies(P):
    say("probe: stream copy of 1 MiB + 16 bytes")
    n = (1 << 20) + 16
    src = torch.randint(0, 1 << 30, (n // 4,), dtype=torch.int32, device="cuda")
    dst = torch.zeros_like(src)
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    assert P.specgen_probe_stream_copy(dst.data_ptr(), src.data_ptr(), n, None) == 0
    assert P.specgen_probe_stream_read(src.data_ptr(), n, sink.data_ptr(), None) == 0
    torch.cuda.synchronize()
    assert torch.equal(dst, src)


@pytest.mark.parametrize("workers", [1, 4, 256])
def test_slice_ring_runs(P, workers):
    say(f"probe: slice ring, 64 blocks x 8 kv heads, 16 tiles per head, {workers} workgroups")
    nblk, hkv, tph = 64, 8, 16
    pool = torch.ones(2 * nblk * hkv * 4096 // 4, dtype=torch.int32, device="cuda")
    kp, vp = pool.data_ptr(), pool.data_ptr() + nblk * hkv * 4096
    ids = np.random.default_rng(3).integers(-5, nblk + 5, size=4 * tph).astype(np.int32)   # some out of the pool
    tab = torch.from_numpy(ids).cuda()
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    assert P.specgen_probe_slice_ring(kp, vp, nblk, hkv, tab.data_ptr(), tph, workers, sink.data_ptr(), None) == 0
    torch.cuda.synchronize()
    assert int(sink.item()) == 0
