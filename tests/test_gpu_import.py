"""KV-block import on the GPU: bit-exact against the oracle's block copy."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_17518_amd as sg
import synth
from gpu_helpers import say

pytestmark = pytest.mark.gpu


def _run(case, bad_expected=0):
    dev = [(torch.from_numpy(case.pool[t].copy()).cuda(), torch.from_numpy(case.staging[t]).cuda(), case.block_bytes)
           for t in range(case.num_tensors)]
    ids = torch.from_numpy(case.dst_ids).cuda()
    bad = torch.zeros(1, dtype=torch.int32, device="cuda")
    sg.specgen_kv_import(dev, ids, case.num_dst_blocks, bad)
    torch.cuda.synchronize()
    assert int(bad.item()) == bad_expected
    for t in range(case.num_tensors):
        ref = case.pool[t].copy()
        assert oracle.kv_import(ref, case.staging[t], case.block_bytes, case.dst_ids, case.num_dst_blocks) == bad_expected
        got = dev[t][0].cpu().numpy()
        assert np.array_equal(got, ref), f"tensor {t} differs at {np.flatnonzero(got != ref)[:8]}"


@pytest.mark.parametrize("n,pool,bb,nt", [(16, 64, 4096, 2), (7, 30, 96, 3), (1, 1, 16, 1), (33, 100, 1028, 4),
                                          (300, 1000, 32768, 2)])
def test_import_bit_exact(n, pool, bb, nt):
    say(f"import n={n} pool={pool} block_bytes={bb} tensors={nt}")
    _run(synth.make_import_case(n=n, num_dst_blocks=pool, block_bytes=bb, num_tensors=nt, seed=n + bb))


def test_import_bad_ids_skipped_and_counted():
    say("import bad ids")
    _run(synth.make_import_case(n=20, num_dst_blocks=50, block_bytes=256, num_tensors=2, seed=3,
                                bad_ids=[0, 5, 19]), bad_expected=3)


def test_import_zero_blocks_is_a_no_op():
    case = synth.make_import_case(n=0, num_dst_blocks=4, block_bytes=64, num_tensors=1, seed=1)
    pool = torch.from_numpy(case.pool[0].copy()).cuda()
    sg.specgen_kv_import([(pool, torch.zeros(16, dtype=torch.uint8, device="cuda"), 64)],
                         torch.zeros(0, dtype=torch.int32, device="cuda"), 4)
    torch.cuda.synchronize()
    assert np.array_equal(pool.cpu().numpy(), case.pool[0])


def test_import_full_size_prefix_restore():
    """2048 prefix blocks of 32 KiB per tensor into a 16384-block pool (K and V)."""
    say("import full size 2048 x 32KiB into 16384")
    case = synth.make_import_case(n=2048, num_dst_blocks=16384, block_bytes=32768, num_tensors=2, seed=3)
    _run(case)
