"""Standalone log-sum-exp merge on the GPU against the oracle's merge."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_17518_amd as sg
from gpu_helpers import say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("S,R,D", [(1, 5, 64), (3, 17, 128), (40, 9, 128), (130, 4, 64), (5, 33, 100)])
@pytest.mark.parametrize("out_dtype", ["fp32", "bf16"])
def test_merge_matches_oracle(S, R, D, out_dtype):
    say(f"merge S={S} R={R} D={D} {out_dtype}")
    rng = np.random.default_rng(S * 100 + R)
    o = rng.standard_normal((S, R, D)).astype(np.float32)
    l = (4 * rng.standard_normal((S, R))).astype(np.float32)
    l[rng.random((S, R)) < 0.2] = -np.inf           # empty parts
    o[np.isinf(l)] = np.nan                          # whose o must be ignored
    if R > 2:
        l[:, 1] = -np.inf                            # a row with only empty parts
    ref, ref_l = oracle.lse_merge(o, l)
    dt = torch.float32 if out_dtype == "fp32" else torch.bfloat16
    out = torch.full((R, D), 7.0, dtype=dt, device="cuda")
    out_l = torch.full((R,), 7.0, dtype=torch.float32, device="cuda")
    sg.specgen_lse_merge(torch.from_numpy(o).cuda(), torch.from_numpy(l).cuda(), out, out_l)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy().astype(np.float64)
    got_l = out_l.cpu().numpy().astype(np.float64)
    assert np.isfinite(got).all()
    if out_dtype == "fp32":
        np.testing.assert_allclose(got, ref, rtol=0, atol=2e-5)
    else:
        np.testing.assert_allclose(got, ref, rtol=2 ** -8, atol=1e-6)
    fin = np.isfinite(ref_l)
    assert np.array_equal(np.isfinite(got_l), fin)
    np.testing.assert_allclose(got_l[fin], ref_l[fin], rtol=0, atol=2e-5)
