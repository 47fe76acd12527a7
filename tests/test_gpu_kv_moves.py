"""KV-block export and per-step append on the GPU: bit-exact against the
oracle's block gather and element copy, and a decode step (append, then
fork-decode attention over the grown suffixes) against the fp64 oracle."""
import copy
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_2606_17518_amd as sg
import synth
from gpu_helpers import check_attn, run_attn, say

pytestmark = pytest.mark.gpu


def _dev(a, dt=None):
    a = np.ascontiguousarray(a)
    return torch.from_numpy(a if dt is None else a.view(dt)).cuda()


# ---- export ------------------------------------------------------------------------

def _export_case(n, pool_blocks, bb, nt, seed, bad=(), repeat=False):
    rng = np.random.default_rng(seed)
    pools = [rng.integers(0, 256, size=pool_blocks * bb, dtype=np.uint8) for _ in range(nt)]
    if repeat:
        ids = rng.integers(0, pool_blocks, size=n).astype(np.int32)
    else:
        ids = rng.permutation(pool_blocks)[:n].astype(np.int32)
    for k, i in enumerate(bad):
        ids[i] = -3 if k % 2 == 0 else pool_blocks + i
    return pools, ids


def _run_export(pools, ids, pool_blocks, bb, bad_expected=0):
    n = ids.size
    dev = [(torch.full((max(n, 1) * bb,), synth.SENTINEL, dtype=torch.uint8, device="cuda"), _dev(p), bb)
           for p in pools]
    bad = torch.zeros(1, dtype=torch.int32, device="cuda")
    sg.specgen_kv_export(dev, _dev(ids), pool_blocks, bad)
    torch.cuda.synchronize()
    assert int(bad.item()) == bad_expected
    for t, p in enumerate(pools):
        ref = np.full(max(n, 1) * bb, synth.SENTINEL, np.uint8)
        assert oracle.kv_export(ref, p, bb, ids, pool_blocks) == bad_expected
        got = dev[t][0].cpu().numpy()
        assert np.array_equal(got, ref), f"tensor {t} differs at {np.flatnonzero(got != ref)[:8]}"


@pytest.mark.parametrize("n,pool,bb,nt", [(16, 64, 4096, 2), (7, 30, 96, 3), (1, 1, 16, 1), (33, 100, 1028, 4),
                                          (300, 1000, 32768, 2)])
def test_export_bit_exact(n, pool, bb, nt):
    say(f"export n={n} pool={pool} block_bytes={bb} tensors={nt}")
    pools, ids = _export_case(n, pool, bb, nt, seed=n + bb)
    _run_export(pools, ids, pool, bb)


def test_export_repeated_and_bad_ids():
    say("export repeated + bad ids")
    pools, ids = _export_case(40, 12, 512, 2, seed=4, bad=[0, 9, 39], repeat=True)
    _run_export(pools, ids, 12, 512, bad_expected=3)


def test_export_zero_blocks_is_a_no_op():
    staging = torch.full((64,), synth.SENTINEL, dtype=torch.uint8, device="cuda")
    pool = torch.zeros(4 * 64, dtype=torch.uint8, device="cuda")
    sg.specgen_kv_export([(staging, pool, 64)], torch.zeros(0, dtype=torch.int32, device="cuda"), 4)
    torch.cuda.synchronize()
    assert bool((staging == synth.SENTINEL).all())


def test_export_then_import_round_trip_full_size():
    """The 2048 prefix blocks (32 KiB per block and tensor, K and V) of a
    16384-block pool migrate out and are restored into other blocks."""
    say("export+import full size 2048 x 32KiB, 16384-block pool")
    bb, nb, n = 32768, 16384, 2048
    pools, ids = _export_case(n, nb, bb, 2, seed=11)
    _run_export(pools, ids, nb, bb)
    rng = np.random.default_rng(12)
    new_ids = rng.permutation(nb)[:n].astype(np.int32)
    dev_pools = [_dev(p) for p in pools]
    staging = [torch.empty(n * bb, dtype=torch.uint8, device="cuda") for _ in pools]
    sg.specgen_kv_export([(s, p, bb) for s, p in zip(staging, dev_pools)], _dev(ids), nb)
    dst = [torch.zeros(nb * bb, dtype=torch.uint8, device="cuda") for _ in pools]
    sg.specgen_kv_import([(d, s, bb) for d, s in zip(dst, staging)], _dev(new_ids), nb)
    torch.cuda.synchronize()
    for t, p in enumerate(pools):
        got = dst[t].cpu().numpy().reshape(nb, bb)
        src = p.reshape(nb, bb)
        assert np.array_equal(got[new_ids], src[ids])


# ---- append ------------------------------------------------------------------------

def _append_dev(b, case, fb, bad=None):
    kvdt = sg.SPECGEN_FP8_E4M3 if b.kv_dtype != "bf16" else sg.SPECGEN_BF16
    el = np.uint8 if b.kv_dtype != "bf16" else np.int16
    sg.specgen_kv_append(fb.k_pool, fb.v_pool, _dev(case.k_new, el), _dev(case.v_new, el), _dev(case.pos),
                         _dev(case.suffix_table_off), _dev(case.suffix_table), b.num_kv_heads, b.head_dim,
                         kv_dtype=kvdt, num_blocks=b.num_blocks, bad_count=bad)


def _check_pools(b, case, fb, bad_expected):
    k, v = b.k_pool.copy(), b.v_pool.copy()
    assert oracle.kv_append(k, v, case.k_new, case.v_new, case.pos, case.suffix_table_off, case.suffix_table,
                            b.num_kv_heads, b.head_dim) == bad_expected
    gk = fb.k_pool.cpu().numpy().view(k.dtype).reshape(k.shape)
    gv = fb.v_pool.cpu().numpy().view(v.dtype).reshape(v.shape)
    assert np.array_equal(gk, k), f"K pool differs in blocks {np.unique(np.nonzero(gk != k)[0])[:8]}"
    assert np.array_equal(gv, v), f"V pool differs in blocks {np.unique(np.nonzero(gv != v)[0])[:8]}"
    return k, v


@pytest.mark.parametrize("kv,D,Hkv", [("bf16", 128, 8), ("bf16", 64, 2), ("fp8_e4m3", 128, 8), ("fp8_e4m3", 64, 4),
                                      ("bf16", 40, 3)])
def test_append_bit_exact(kv, D, Hkv):
    """Suffix lengths 0, multiples of 16 (fresh blocks) and ragged ones; two
    bad forks (no table entry for the position; an id outside the pool)."""
    say(f"append kv={kv} D={D} Hkv={Hkv}")
    S = [0, 16, 5, 33, 48, 1, 15, 200, 17, 64]
    b = synth.make_fork_batch(prefix_lens=[70], forks_per_trace=len(S), suffix_lens=S, num_q_heads=Hkv * 2,
                              num_kv_heads=Hkv, head_dim=D, kv_dtype=kv, seed=D + Hkv)
    case = synth.make_append_case(b, seed=5, bad_forks=[3, 8])
    fb = sg.ForkBatchTensors.from_numpy(b)
    bad = torch.zeros(1, dtype=torch.int32, device="cuda")
    _append_dev(b, case, fb, bad)
    torch.cuda.synchronize()
    assert int(bad.item()) == 2
    _check_pools(b, case, fb, 2)


def _step_batch(b, case, k, v):
    """The batch after the append step, on the host: grown suffixes, the new
    tables, the appended pools; fresh E4M3 blocks get a scale."""
    b2 = copy.copy(b)
    b2.k_pool, b2.v_pool = k, v
    b2.suffix_len = (case.pos + 1).astype(np.int32)
    b2.suffix_table_off, b2.suffix_table = case.suffix_table_off, case.suffix_table
    if b.kv_dtype != "bf16":
        b2.k_scale, b2.v_scale = b.k_scale.copy(), b.v_scale.copy()
        used = np.isfinite(b.k_scale)
        b2.k_scale[case.fresh_blocks] = np.float32(b.k_scale[used].mean())
        b2.v_scale[case.fresh_blocks] = np.float32(b.v_scale[used].mean())
    return b2


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_decode_step_append_then_attend(kv):
    """Append each fork's token with the GPU, then attend over S_f + 1 tokens;
    the result matches the oracle's attention over the oracle-appended pools."""
    say(f"decode step append+attend kv={kv}")
    S = [0, 16, 31, 32, 100, 7]
    b = synth.make_fork_batch(prefix_lens=[300], forks_per_trace=len(S), suffix_lens=S, num_q_heads=16,
                              num_kv_heads=2, head_dim=128, kv_dtype=kv, seed=77)
    case = synth.make_append_case(b, seed=8)
    assert case.fresh_blocks.size == 3
    fb = sg.ForkBatchTensors.from_numpy(b)
    _append_dev(b, case, fb)
    torch.cuda.synchronize()
    k, v = _check_pools(b, case, fb, 0)
    b2 = _step_batch(b, case, k, v)
    fb2 = dataclasses.replace(fb, suffix_len=_dev(b2.suffix_len), suffix_table_off=_dev(b2.suffix_table_off),
                              suffix_table=_dev(b2.suffix_table), suffix_len_h=b2.suffix_len.copy(),
                              suffix_table_off_h=b2.suffix_table_off.copy())
    if kv != "bf16":
        fb2 = dataclasses.replace(fb2, k_scale=_dev(b2.k_scale), v_scale=_dev(b2.v_scale))
    o, l = run_attn(b2, fb=fb2)
    ro, rl = oracle.fork_decode_attn(b2)
    check_attn(o, ro, l, rl, what=f"append+attend {kv}")


def test_append_full_size_trace_p32k_f16():
    """16 forks of one 32768-token trace, 8 kv heads, D = 128, 16384-block
    pool: every fork's next token, byte-exact over the whole pools."""
    say("append full size trace_p32k_f16")
    b = synth.workload("trace_p32k_f16")
    case = synth.make_append_case(b, seed=3)
    fb = sg.ForkBatchTensors.from_numpy(b)
    _append_dev(b, case, fb)
    torch.cuda.synchronize()
    _check_pools(b, case, fb, 0)
