"""The Python binding's checks of the tensors it hands to the library (CPU,
no GPU needed: every case is rejected before any library call).  The C ABI
receives bare pointers, so an output or staging buffer shorter than the call's
extent would otherwise become an out-of-bounds access on the device."""
import numpy as np
import pytest
import torch

import paper_2606_17518_amd as sg
import paper_2606_17518_amd.binding as B
import synth


@pytest.fixture(scope="module")
def batch():
    b = synth.make_fork_batch(prefix_lens=[100], forks_per_trace=3, suffix_lens=[5, 20, 40], num_q_heads=8,
                              num_kv_heads=2, head_dim=64, seed=5)
    s, keep = B.host_batch_struct(b)
    return b, s, keep


def _ws():
    return torch.zeros(64, dtype=torch.float32)


def test_decode_outputs_checked(batch):
    b, s, _ = batch
    N, Hq, D = b.num_forks, b.num_q_heads, b.head_dim
    with pytest.raises(ValueError, match="out holds"):
        sg.specgen_fork_decode_attn(s, torch.empty(N * Hq * D - 1, dtype=torch.bfloat16), None, _ws())
    with pytest.raises(ValueError, match="out: dtype"):
        sg.specgen_fork_decode_attn(s, torch.empty((N, Hq, D), dtype=torch.float32), None, _ws())
    with pytest.raises(ValueError, match="contiguous"):
        sg.specgen_fork_decode_attn(s, torch.empty((N, D, Hq), dtype=torch.bfloat16).transpose(1, 2), None, _ws())
    with pytest.raises(ValueError, match="out_lse holds"):
        sg.specgen_fork_decode_attn(s, torch.empty((N, Hq, D), dtype=torch.bfloat16),
                                    torch.empty((N, Hq - 1), dtype=torch.float32), _ws())
    # right size and dtype, but host memory
    with pytest.raises(ValueError, match="device memory"):
        sg.specgen_fork_decode_attn(s, torch.empty((N, Hq, D), dtype=torch.bfloat16), None, _ws())
    with pytest.raises(ValueError, match="out holds"):
        sg.specgen_fork_decode_attn_noalloc(s, torch.empty((N - 1, Hq, D), dtype=torch.bfloat16), None)
    with pytest.raises(ValueError, match="out_lse holds"):
        sg.specgen_fork_decode_attn_phase(s, sg.SPECGEN_PHASE_MERGE, torch.empty((N, Hq, D), dtype=torch.bfloat16),
                                          torch.empty(1, dtype=torch.float32), _ws())


def test_prefill_outputs_need_a_row_per_query(batch):
    """A prefill writes sum(q_len) rows, not one per fork."""
    b, s, _ = batch
    q_len = np.array([2, 5, 9], np.int32)
    N, Hq, D = b.num_forks, b.num_q_heads, b.head_dim
    with pytest.raises(ValueError, match="out holds"):
        sg.specgen_fork_prefill_attn(s, q_len, torch.empty((N, Hq, D), dtype=torch.bfloat16), None, _ws())
    Q = int(q_len.sum())
    with pytest.raises(ValueError, match="out_lse holds"):
        sg.specgen_fork_prefill_attn(s, q_len, torch.empty((Q, Hq, D), dtype=torch.bfloat16),
                                     torch.empty((N, Hq), dtype=torch.float32), _ws())
    with pytest.raises(ValueError, match="device memory"):
        sg.specgen_fork_prefill_attn(s, q_len, torch.empty((Q, Hq, D), dtype=torch.bfloat16),
                                     torch.empty((Q, Hq), dtype=torch.float32), _ws())


def test_merge_buffers_checked():
    S, R, D = 3, 5, 64
    o, l = torch.zeros((S, R, D), dtype=torch.float32), torch.zeros((S, R), dtype=torch.float32)
    with pytest.raises(ValueError, match="o_parts: dtype"):
        sg.specgen_lse_merge(o.half(), l, torch.empty((R, D), dtype=torch.float32))
    with pytest.raises(ValueError, match="out holds"):
        sg.specgen_lse_merge(o, l, torch.empty((R - 1, D), dtype=torch.bfloat16))
    with pytest.raises(ValueError, match="out_lse holds"):
        sg.specgen_lse_merge(o, l, torch.empty((R, D), dtype=torch.float32), torch.empty(R - 1, dtype=torch.float32))


def test_block_move_buffers_checked():
    bb, n, nb = 64, 4, 10
    ids = torch.arange(n, dtype=torch.int32)
    pool, staging = torch.zeros(nb * bb, dtype=torch.uint8), torch.zeros(n * bb, dtype=torch.uint8)
    with pytest.raises(ValueError, match="src_staging holds"):
        sg.specgen_kv_import([(pool, staging[:-1], bb)], ids, nb)
    with pytest.raises(ValueError, match="dst_pool holds"):
        sg.specgen_kv_import([(pool[:-bb], staging, bb)], ids, nb)
    with pytest.raises(ValueError, match="dst_block_ids: dtype"):
        sg.specgen_kv_import([(pool, staging, bb)], ids.long(), nb)
    with pytest.raises(ValueError, match="dst_staging holds"):
        sg.specgen_kv_export([(staging[:bb], pool, bb)], ids, nb)
    with pytest.raises(ValueError, match="src_pool holds"):
        sg.specgen_kv_export([(staging, pool, bb)], ids, nb + 1)


def test_append_buffers_checked():
    N, H, D, nb = 3, 2, 64, 8
    blk = H * 16 * D
    pools = [torch.zeros(nb * blk, dtype=torch.bfloat16) for _ in range(2)]
    new = [torch.zeros((N, H, D), dtype=torch.bfloat16) for _ in range(2)]
    pos = torch.zeros(N, dtype=torch.int32)
    off = torch.arange(N + 1, dtype=torch.int32)
    tab = torch.zeros(N, dtype=torch.int32)
    with pytest.raises(ValueError, match="k_new holds"):
        sg.specgen_kv_append(pools[0], pools[1], new[0][:-1], new[1], pos, off, tab, H, D)
    with pytest.raises(ValueError, match="suffix_table_off holds"):
        sg.specgen_kv_append(pools[0], pools[1], new[0], new[1], pos, off[:-1], tab, H, D)
    with pytest.raises(ValueError, match="k_pool holds"):
        sg.specgen_kv_append(pools[0], pools[1], new[0], new[1], pos, off, tab, H, D, num_blocks=nb + 1)
    with pytest.raises(ValueError, match="pos: dtype"):
        sg.specgen_kv_append(pools[0], pools[1], new[0], new[1], pos.long(), off, tab, H, D)
    with pytest.raises(ValueError, match="device memory"):
        sg.specgen_kv_append(pools[0], pools[1], new[0], new[1], pos, off, tab, H, D)
