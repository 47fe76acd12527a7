"""The C-ABI library on a host without a GPU: it loads, exports every entry
point include/specgen.h declares, and rejects bad arguments before touching
the device (these calls return during argument checking)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "specgen.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(specgen_\w+)\s*\(", src)))


@pytest.fixture(scope="module")
def L():
    import paper_2606_17518_amd as sg
    lib_path = os.path.join(ROOT, "paper_2606_17518_amd", "libspecgen.so")
    if not os.path.exists(lib_path):
        sg.build.build()
    return sg.lib()


def test_every_declared_symbol_is_exported(L):
    names = _declared()
    assert set(names) == {"specgen_fork_decode_attn_workspace_size", "specgen_fork_decode_attn",
                          "specgen_fork_decode_attn_phase", "specgen_fork_prefill_attn_workspace_size",
                          "specgen_fork_prefill_attn", "specgen_kv_import", "specgen_kv_export",
                          "specgen_kv_append", "specgen_lse_merge", "specgen_last_error",
                          "specgen_fork_decode_attn_split", "specgen_fork_decode_attn_noalloc"}
    for n in names:
        assert hasattr(L, n), n


def _host_batch(**kw):
    import paper_2606_17518_amd.binding as B
    s = B.ForkBatchC()
    s.num_traces, s.num_forks, s.num_q_heads, s.num_kv_heads, s.head_dim, s.block_size = 1, 2, 8, 2, 64, 16
    s.num_blocks, s.sm_scale, s.kv_dtype, s.path, s.flags = 8, 0.125, 0, 0, 0
    fake = 0x10000   # never dereferenced: every call below fails argument checks first
    for f in ("q", "k_pool", "v_pool", "fork_off", "prefix_len", "prefix_table_off", "prefix_table",
              "suffix_len", "suffix_table_off", "suffix_table"):
        setattr(s, f, fake)
    keep = [np.array([0, 2], np.int32), np.array([20], np.int32), np.array([3, 0], np.int32),
            np.array([0, 2], np.int32), np.array([0, 1, 1], np.int32)]
    s.fork_off_h, s.prefix_len_h, s.suffix_len_h, s.prefix_table_off_h, s.suffix_table_off_h = \
        (a.ctypes.data for a in keep)
    for k, v in kw.items():
        setattr(s, k, v)
    return s, keep


@pytest.mark.parametrize("field,value,status", [
    ("num_traces", 0, 1), ("num_forks", 0, 1), ("num_q_heads", 7, 1), ("head_dim", 96, 2),
    ("block_size", 32, 2), ("sm_scale", 0.0, 1), ("sm_scale", float("nan"), 1), ("kv_dtype", 5, 2),
    ("path", 9, 1), ("flags", 2, 1), ("flags", 1, 1), ("q", None, 1), ("suffix_len_h", None, 1), ("num_blocks", 0, 1),
    ("suffix_table_off_h", None, 1), ("prefix_table_off_h", None, 1),
])
def test_bad_batch_rejected_without_launch(L, field, value, status):
    s, keep = _host_batch(**{field: value})
    n = C.c_size_t(123)
    assert L.specgen_fork_decode_attn_workspace_size(C.byref(s), C.byref(n)) == status
    assert n.value == 123
    assert L.specgen_last_error().decode() != ""
    assert L.specgen_fork_decode_attn(C.byref(s), C.c_void_p(0x10000), None, None, 0, None) == status
    for phase in (0, 1, 2):
        assert L.specgen_fork_decode_attn_phase(C.byref(s), phase, C.c_void_p(0x10000), None, None, 0, None) == status


def test_bad_lengths_rejected(L):
    import paper_2606_17518_amd.binding as B
    s, keep = _host_batch()
    bad = np.array([0, 3], np.int32)          # fork_off must end at N = 2
    s.fork_off_h = bad.ctypes.data
    n = C.c_size_t(0)
    assert L.specgen_fork_decode_attn_workspace_size(C.byref(s), C.byref(n)) == B.SPECGEN_ERR_INVALID_ARG
    s, keep = _host_batch()
    neg = np.array([-1, 0], np.int32)
    s.suffix_len_h = neg.ctypes.data
    assert L.specgen_fork_decode_attn_workspace_size(C.byref(s), C.byref(n)) == B.SPECGEN_ERR_INVALID_ARG
    zero_prefix = np.array([0], np.int32)
    s, keep = _host_batch()
    s.prefix_len_h = zero_prefix.ctypes.data
    assert L.specgen_fork_decode_attn_workspace_size(C.byref(s), C.byref(n)) == B.SPECGEN_ERR_INVALID_ARG


def test_import_and_merge_argument_errors(L):
    import paper_2606_17518_amd.binding as B
    t = (B.KvTensorC * 1)()
    t[0].dst_pool, t[0].src_staging, t[0].block_bytes = 0x10000, 0x20000, 6
    assert L.specgen_kv_import(t, 1, C.c_void_p(0x30000), 4, 16, None, None) == B.SPECGEN_ERR_INVALID_ARG
    t[0].block_bytes = 64
    assert L.specgen_kv_import(t, 0, C.c_void_p(0x30000), 4, 16, None, None) == B.SPECGEN_ERR_INVALID_ARG
    assert L.specgen_kv_import(t, 5, C.c_void_p(0x30000), 4, 16, None, None) == B.SPECGEN_ERR_INVALID_ARG
    assert L.specgen_kv_import(t, 1, None, 4, 16, None, None) == B.SPECGEN_ERR_INVALID_ARG
    assert L.specgen_kv_import(t, 1, C.c_void_p(0x30000), -1, 16, None, None) == B.SPECGEN_ERR_INVALID_ARG
    P = C.c_void_p(0x10000)
    assert L.specgen_lse_merge(P, P, 0, 4, 64, P, 0, None, None) == B.SPECGEN_ERR_INVALID_ARG
    assert L.specgen_lse_merge(P, P, 2, 4, 2000, P, 0, None, None) == B.SPECGEN_ERR_INVALID_ARG
    assert L.specgen_lse_merge(P, P, 2, 4, 64, P, 7, None, None) == B.SPECGEN_ERR_INVALID_ARG


def test_export_argument_errors(L):
    import paper_2606_17518_amd.binding as B
    t = (B.KvExportTensorC * 1)()
    t[0].dst_staging, t[0].src_pool, t[0].block_bytes = 0x10000, 0x20000, 6
    ids = C.c_void_p(0x30000)
    assert L.specgen_kv_export(t, 1, ids, 4, 16, None, None) == B.SPECGEN_ERR_INVALID_ARG
    t[0].block_bytes = 64
    assert L.specgen_kv_export(None, 1, ids, 4, 16, None, None) == B.SPECGEN_ERR_INVALID_ARG
    assert L.specgen_kv_export(t, 0, ids, 4, 16, None, None) == B.SPECGEN_ERR_INVALID_ARG
    assert L.specgen_kv_export(t, 5, ids, 4, 16, None, None) == B.SPECGEN_ERR_INVALID_ARG
    assert L.specgen_kv_export(t, 1, None, 4, 16, None, None) == B.SPECGEN_ERR_INVALID_ARG
    assert L.specgen_kv_export(t, 1, ids, -1, 16, None, None) == B.SPECGEN_ERR_INVALID_ARG
    assert L.specgen_kv_export(t, 1, ids, 4, -1, None, None) == B.SPECGEN_ERR_INVALID_ARG
    t[0].src_pool = 0x20008      # not 16-byte aligned for a 64-byte block
    assert L.specgen_kv_export(t, 1, ids, 4, 16, None, None) == B.SPECGEN_ERR_INVALID_ARG
    t[0].dst_staging = 0
    assert L.specgen_kv_export(t, 1, ids, 4, 16, None, None) == B.SPECGEN_ERR_INVALID_ARG
    # n = 0 queues nothing, so it succeeds without touching the device
    t[0].dst_staging, t[0].src_pool = 0x10000, 0x20000
    assert L.specgen_kv_export(t, 1, None, 0, 16, None, None) == B.SPECGEN_OK


def _append_desc(**kw):
    import paper_2606_17518_amd.binding as B
    a = B.KvAppendC(num_forks=2, num_kv_heads=2, head_dim=64, kv_dtype=B.SPECGEN_BF16, num_blocks=8)
    for f in ("k_pool", "v_pool", "k_new", "v_new", "pos", "suffix_table_off", "suffix_table"):
        setattr(a, f, 0x10000)
    for k, v in kw.items():
        setattr(a, k, v)
    return a


@pytest.mark.parametrize("field,value,status", [
    ("num_forks", -1, 1), ("num_kv_heads", 0, 1), ("head_dim", 0, 1), ("head_dim", 1025, 1), ("kv_dtype", 2, 2),
    ("kv_dtype", 7, 2), ("num_blocks", 0, 1), ("k_new", None, 1), ("suffix_table", None, 1), ("pos", None, 1),
    ("v_pool", 0x10001, 1),
])
def test_append_argument_errors(L, field, value, status):
    a = _append_desc(**{field: value})
    assert L.specgen_kv_append(C.byref(a), None) == status
    assert L.specgen_last_error().decode() != ""


def test_append_null_and_empty(L):
    import paper_2606_17518_amd.binding as B
    assert L.specgen_kv_append(None, None) == B.SPECGEN_ERR_INVALID_ARG
    # no forks: nothing is queued, pointers are not needed
    a = B.KvAppendC(num_forks=0, num_kv_heads=1, head_dim=64, kv_dtype=B.SPECGEN_FP8_E4M3, num_blocks=1)
    assert L.specgen_kv_append(C.byref(a), None) == B.SPECGEN_OK
    # 1-byte elements need no alignment
    a = _append_desc(kv_dtype=B.SPECGEN_FP8_E4M3, num_forks=0, v_pool=0x10001)
    assert L.specgen_kv_append(C.byref(a), None) == B.SPECGEN_OK


def _tree_batch(parent, forks=1, P=20):
    """T traces with `forks` forks each (no suffixes) and the given parents."""
    import paper_2606_17518_amd.binding as B
    T = len(parent)
    s, keep = _host_batch()
    N = T * forks
    arrs = [np.arange(0, N + 1, forks, dtype=np.int32), np.full(T, P, np.int32), np.zeros(N, np.int32),
            np.arange(0, T + 1, dtype=np.int32) * ((P + 15) // 16), np.zeros(N + 1, np.int32),
            np.asarray(parent, np.int32)]
    keep += arrs
    s.num_traces, s.num_forks = T, N
    s.fork_off_h, s.prefix_len_h, s.suffix_len_h, s.prefix_table_off_h, s.suffix_table_off_h, s.prefix_parent_h = \
        (a.ctypes.data for a in arrs)
    return s, keep


@pytest.mark.parametrize("parent,status", [
    ([-1, 0, 1], 0), ([-1, 0, 0, 2, -1, 4], 0), ([-1, -1], 0),
    ([0], 1), ([-1, 1], 1), ([-1, 2, 0], 1), ([-2], 1),
    ([-1, 0, -1, 1], 1),                    # 1 is not an ancestor of trace 2 (not depth-first)
    ([-1] + list(range(8)), 2),             # a chain of 9 traces
    ([-1] + list(range(7)), 0),             # a chain of 8 traces
])
def test_nested_prefix_parents_validated(L, parent, status):
    s, keep = _tree_batch(parent)
    n = C.c_size_t(0)
    assert L.specgen_fork_decode_attn_workspace_size(C.byref(s), C.byref(n)) == status, \
        L.specgen_last_error().decode()
    if status == 0:
        assert n.value > 0


def test_prefill_q_len_validated(L):
    import paper_2606_17518_amd.binding as B
    s, keep = _host_batch()             # suffix lengths 3 and 0
    n = C.c_size_t(7)
    for ql, status in (([1, 1], 1), ([0, 0], 1), ([4, 0], 1), (None, 1)):
        arr = None if ql is None else np.array(ql, np.int32)
        p = None if arr is None else arr.ctypes.data_as(C.c_void_p)
        assert L.specgen_fork_prefill_attn_workspace_size(C.byref(s), p, C.byref(n)) == status
        assert L.specgen_fork_prefill_attn(C.byref(s), p, C.c_void_p(0x10000), None, None, 0, None) == status
    assert n.value == 7
    s2, keep2 = _host_batch()
    ql = np.array([3, 2], np.int32)
    suf = np.array([3, 2], np.int32)
    soff = np.array([0, 1, 2], np.int32)
    keep2 += [suf, soff]
    s2.suffix_len_h, s2.suffix_table_off_h = suf.ctypes.data, soff.ctypes.data
    assert L.specgen_fork_prefill_attn_workspace_size(C.byref(s2), ql.ctypes.data_as(C.c_void_p), C.byref(n)) == 0
    assert n.value > 0
    # more than 512 queries in one call
    s3, keep3 = _host_batch()
    big = np.array([600, 1], np.int32)
    boff = np.array([0, 38, 39], np.int32)
    s3.suffix_len_h, s3.suffix_table_off_h = big.ctypes.data, boff.ctypes.data
    ql3 = np.array([600, 1], np.int32)
    assert L.specgen_fork_prefill_attn_workspace_size(C.byref(s3), ql3.ctypes.data_as(C.c_void_p), C.byref(n)) == 2


@pytest.mark.parametrize("fork_off,parent,status", [
    ([0, 0, 2], [-1, 0], 0),        # the root has no forks of its own, its child has two
    ([0, 2, 2], [-1, 0], 1),        # an empty leaf
    ([0, 0, 2], [-1, -1], 1),       # an empty root with nothing below it
])
def test_trace_without_own_forks(L, fork_off, parent, status):
    s, keep = _tree_batch(parent, forks=1)
    fo = np.array(fork_off, np.int32)
    keep.append(fo)
    s.fork_off_h = fo.ctypes.data
    n = C.c_size_t(0)
    assert L.specgen_fork_decode_attn_workspace_size(C.byref(s), C.byref(n)) == status, \
        L.specgen_last_error().decode()


@pytest.mark.parametrize("which,off,lens,status", [
    ("prefix", [-100000, 2], None, 1),           # negative start
    ("prefix", [0, 1], None, 1),                 # 20 prefix tokens need 2 ids
    ("prefix", [3, 5], None, 0),                 # any start, enough ids
    ("suffix", [0, 0, 0], None, 1),              # fork 0 has 3 tokens and no id
    ("suffix", [0, 1, 0], None, 1),              # decreasing
    ("suffix", [-1, 0, 0], None, 1),             # negative start
    ("suffix", [4, 5, 5], None, 0),
    ("suffix", [0, 1, 1], [17, 0], 1),           # 17 tokens need 2 ids
    ("suffix", [0, 2, 2], [17, 0], 0),
    ("suffix", [0, 2, 2], [17, 1], 1),           # fork 1's one token needs one id
])
def test_table_offsets_validated(L, which, off, lens, status):
    """Offset mirrors that would make the kernels read past a fork's or trace's
    ids are rejected before any launch (decode and prefill entry points)."""
    s, keep = _host_batch()
    o = np.array(off, np.int32)
    keep.append(o)
    setattr(s, f"{which}_table_off_h", o.ctypes.data)
    if lens is not None:
        ln = np.array(lens, np.int32)
        keep.append(ln)
        s.suffix_len_h = ln.ctypes.data
    n = C.c_size_t(5)
    assert L.specgen_fork_decode_attn_workspace_size(C.byref(s), C.byref(n)) == status, L.specgen_last_error().decode()
    if status:
        assert n.value == 5
        assert "table_off" in L.specgen_last_error().decode()
        assert L.specgen_fork_decode_attn(C.byref(s), C.c_void_p(0x10000), None, None, 0, None) == status
        ql = np.ones(2, np.int32)
        assert L.specgen_fork_prefill_attn_workspace_size(C.byref(s), ql.ctypes.data_as(C.c_void_p),
                                                          C.byref(n)) == status


@pytest.mark.parametrize("T,N,status", [(32, 512, 0), (33, 33, 2), (1, 513, 2), (32, 513, 2)])
def test_traces_and_forks_per_call(L, T, N, status):
    """At most 32 traces and 512 forks per call; a larger batch is
    SPECGEN_ERR_UNSUPPORTED before any launch (forks spread over the traces as
    evenly as they go, 20 prefix tokens per trace, 3 suffix tokens per fork)."""
    fork_off = np.array([(t * N) // T for t in range(T + 1)], np.int32)
    plen = np.full(T, 20, np.int32)
    pto = np.arange(T + 1, dtype=np.int32) * 2
    slen = np.full(N, 3, np.int32)
    sto = np.arange(N + 1, dtype=np.int32)
    s, keep = _host_batch(num_traces=T, num_forks=N)
    keep += [fork_off, plen, pto, slen, sto]
    s.fork_off_h, s.prefix_len_h, s.prefix_table_off_h = fork_off.ctypes.data, plen.ctypes.data, pto.ctypes.data
    s.suffix_len_h, s.suffix_table_off_h = slen.ctypes.data, sto.ctypes.data
    n = C.c_size_t(7)
    assert L.specgen_fork_decode_attn_workspace_size(C.byref(s), C.byref(n)) == status, L.specgen_last_error().decode()
    if status:
        assert n.value == 7
        assert "per call" in L.specgen_last_error().decode()
        assert L.specgen_fork_decode_attn(C.byref(s), C.c_void_p(0x10000), None, None, 0, None) == status
    else:
        assert n.value > 0


@pytest.mark.parametrize("path", ["auto", "mfma", "dot"])
def test_split_query_tiles_every_item_once(L, path):
    """specgen_fork_decode_attn_split (host only): the segments of every work
    item cover its keys exactly once, in worker order, and its rows are the
    trace's (or group's) rows cut into row blocks."""
    import synth
    import paper_2606_17518_amd as sg
    b = synth.make_fork_batch(prefix_lens=[5000, 37], forks_per_trace=[20, 3], suffix_range=(0, 700),
                              num_q_heads=16, num_kv_heads=2, head_dim=128, seed=3)
    sp = sg.specgen_fork_decode_attn_split(b, path)
    g = b.group
    items = {}
    for k in range(len(sp["kind"])):
        key = (int(sp["kind"][k]), int(sp["trace"][k]), int(sp["fork"][k]), int(sp["kv_head"][k]), int(sp["row_block"][k]))
        items.setdefault(key, []).append((int(sp["kernel"][k]), int(sp["worker"][k]), int(sp["first_token"][k]),
                                          int(sp["num_tokens"][k]), int(sp["first_row"][k]), int(sp["num_rows"][k])))
    rows_seen = {}
    for (kind, t, f, j, rb), segs in items.items():
        segs.sort(key=lambda s: s[1])
        assert len({s[0] for s in segs}) == 1                      # one kernel per item
        n = int(b.prefix_len[t]) if kind == 0 else int(b.suffix_len[f])
        pos = 0
        for s in segs:
            assert s[2] == pos and s[3] > 0
            pos += s[3]
        assert pos == n
        assert len({(s[4], s[5]) for s in segs}) == 1
        r0, nr = segs[0][4], segs[0][5]
        rows_seen.setdefault((kind, t, f, j), []).append((r0, nr))
        if path == "dot" or (path == "auto" and kind == 0 and (b.fork_off[t + 1] - b.fork_off[t]) * g < 16):
            assert segs[0][0] == 1
    for (kind, t, f, j), blocks in rows_seen.items():
        total = (b.fork_off[t + 1] - b.fork_off[t]) * g if kind == 0 else g
        blocks.sort()
        assert blocks[0][0] == 0 and sum(nr for _, nr in blocks) == total
    # every prefix item and every non-empty suffix item appears
    assert {(k[1], k[3]) for k in items if k[0] == 0} == {(t, j) for t in range(2) for j in range(2)}
    assert {(k[2], k[3]) for k in items if k[0] == 1} == {(f, j) for f in range(b.num_forks) if b.suffix_len[f] > 0
                                                         for j in range(2)}



def test_probe_library_exports_its_header():
    """libspecgen_probe.so (the benchmark's memory ceilings) exports every call
    include/specgen_probe.h declares, and rejects bad sizes without a launch."""
    import ctypes
    from paper_2606_17518_amd.build import PROBE_LIB_PATH
    src = open(os.path.join(ROOT, "include", "specgen_probe.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = sorted(set(re.findall(r"\b(specgen_probe_\w+)\s*\(", src)))
    assert names == ["specgen_probe_slice_ring", "specgen_probe_stream_copy", "specgen_probe_stream_read"]
    lib = ctypes.CDLL(PROBE_LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    lib.specgen_probe_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
    lib.specgen_probe_stream_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    assert lib.specgen_probe_stream_read(0x10000, 24, 0x20000, None) == 1      # not a multiple of 16
    assert lib.specgen_probe_stream_copy(0x10000, None, 64, None) == 1
    ring = lib.specgen_probe_slice_ring
    ring.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
                     ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    ok = (0x10000, 0x20000, 64, 8, 0x30000, 16, 4, 0x40000, None)
    for i, bad in [(0, None), (1, 0x20008), (2, 0), (3, 0), (4, None), (5, 0), (6, 0), (7, None)]:
        args = list(ok)
        args[i] = bad
        assert ring(*args) == 1, (i, bad)
    # a share of more than 1024 tiles per workgroup: 8 heads x 2048 tiles on 8 workgroups
    assert ring(0x10000, 0x20000, 64, 8, 0x30000, 2048, 8, 0x40000, None) == 1


def test_noalloc_scratch_size_and_rejection(L):
    """The no-allocation entry point's scratch size is the header's, and a batch
    needing more workspace is rejected during argument checking (no device
    work: this runs without a GPU)."""
    import re
    import types
    import paper_2606_17518_amd as sg
    hdr = open(os.path.join(ROOT, "include", "specgen.h")).read()
    m = re.search(r"#define SPECGEN_NOALLOC_SCRATCH_BYTES \((\d+)ull << (\d+)\)", hdr)
    assert m and int(m.group(1)) << int(m.group(2)) == sg.SPECGEN_NOALLOC_SCRATCH_BYTES
    P, N = 131072, 32
    o = types.SimpleNamespace(num_traces=1, num_forks=N, num_q_heads=128, num_kv_heads=8, head_dim=128,
                              num_blocks=10 ** 6, sm_scale=0.1, kv_dtype="fp8_e4m3", fork_off=[0, N], prefix_len=[P],
                              suffix_len=[300] * N, prefix_table_off=[0, P // 16],
                              suffix_table_off=list(range(0, 19 * (N + 1), 19)))
    s, keep = sg.host_batch_struct(o)
    for f in ("q", "k_pool", "v_pool", "k_scale", "v_scale", "fork_off", "prefix_len", "prefix_table_off",
              "prefix_table", "suffix_len", "suffix_table_off", "suffix_table"):
        setattr(s, f, 0x10000)
    n = C.c_size_t(0)
    assert L.specgen_fork_decode_attn_workspace_size(C.byref(s), C.byref(n)) == 0
    assert n.value > sg.SPECGEN_NOALLOC_SCRATCH_BYTES
    assert L.specgen_fork_decode_attn_noalloc(C.byref(s), C.c_void_p(0x10000), None, None) == 3
    assert "scratch" in L.specgen_last_error().decode()
    bad, keep2 = sg.host_batch_struct(o)   # NULL device pointers: rejected first
    assert L.specgen_fork_decode_attn_noalloc(C.byref(bad), C.c_void_p(0x10000), None, None) == 1


def test_fp8_scores_flag_validated(L):
    """SPECGEN_FLAG_FP8_SCORES: E4M3 KV with head_dim 128 only."""
    import paper_2606_17518_amd.binding as B
    n = C.c_size_t(0)
    s, keep = _host_batch(flags=B.SPECGEN_FLAG_FP8_SCORES, kv_dtype=B.SPECGEN_FP8_E4M3, k_scale=0x10000, v_scale=0x10000)
    assert L.specgen_fork_decode_attn_workspace_size(C.byref(s), C.byref(n)) == B.SPECGEN_ERR_UNSUPPORTED   # D = 64
    s.head_dim = 128
    assert L.specgen_fork_decode_attn_workspace_size(C.byref(s), C.byref(n)) == 0
    s.kv_dtype = B.SPECGEN_BF16
    assert L.specgen_fork_decode_attn_workspace_size(C.byref(s), C.byref(n)) == B.SPECGEN_ERR_INVALID_ARG
    assert "E4M3" in L.specgen_last_error().decode()


def test_debug_library_exports_the_same_entry_points(L):
    """libspecgen_debug.so (SPECGEN_DEBUG_CHECKS) is a drop-in build of the
    library: every declared entry point, and the same argument checks."""
    import paper_2606_17518_amd.binding as B
    D = B.debug_lib()
    for n in _declared():
        assert hasattr(D, n), n
    s, keep = _host_batch(num_traces=0)
    n = C.c_size_t(0)
    assert D.specgen_fork_decode_attn_workspace_size(C.byref(s), C.byref(n)) == 1
    assert b"num_traces" in D.specgen_last_error()


def test_timeline_library_exports_its_header_and_the_entry_points(L):
    """libspecgen_timeline.so (the partial kernel built with per-slot clock
    stamps) is a drop-in build of the library that also exports every call of
    include/specgen_timeline.h, which the release library does not."""
    import paper_2606_17518_amd.binding as B
    T = B.timeline_lib()
    for n in _declared():
        assert hasattr(T, n), n
    src = open(os.path.join(ROOT, "include", "specgen_timeline.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = sorted(set(re.findall(r"\b(specgen_timeline_\w+)\s*\(", src)))
    assert names == ["specgen_timeline_clear", "specgen_timeline_read", "specgen_timeline_shape"]
    for n in names:
        assert hasattr(T, n), n
        assert not hasattr(L, n), n
    w, k = C.c_int(0), C.c_int(0)
    assert T.specgen_timeline_shape(C.byref(w), C.byref(k)) == 0
    assert (w.value, k.value) == (2048, 128)
    assert T.specgen_timeline_shape(None, C.byref(k)) == 1
    assert T.specgen_timeline_read(None, None) == 1
    s, keep = _host_batch(num_traces=0)
    n = C.c_size_t(0)
    assert T.specgen_fork_decode_attn_workspace_size(C.byref(s), C.byref(n)) == 1


def test_lds_layouts_of_the_partial_kernel(tmp_path):
    """The partial kernel's LDS placements (csrc/lds_layout.h), driven by a g++
    harness: the V^T placement fills every slot once and its DMA inverse stays
    inside each 1 KiB piece; operand reads are conflict-free under every lane
    grouping that fits the LDS measurements; the E4M3 K decode covers each
    (row, chunk pair) once on distinct bank groups per write pass."""
    import subprocess
    exe = str(tmp_path / "lds_layout_check")
    subprocess.run(["g++", "-O1", "-std=c++17", "-Wall", "-Werror", "-o", exe,
                    os.path.join(ROOT, "tests", "lds_layout_check.cpp")], check=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all layout checks passed" in r.stdout


def test_debug_block_id_check_on_host_tables(tmp_path):
    """The debug build's block-id check (csrc/table_check.h), driven with host
    tables by a g++ harness: ids past ceil(len/16) are never read, -1 and
    num_blocks are caught in either table, prefill traces whose prefix lives in
    the suffix table are checked there, and empty suffixes read nothing."""
    import subprocess
    exe = str(tmp_path / "table_check")
    subprocess.run(["g++", "-O1", "-std=c++17", "-Wall", "-Werror", "-o", exe,
                    os.path.join(ROOT, "tests", "table_check_driver.cpp")], check=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all table checks passed" in r.stdout


def test_concurrent_host_calls(L):
    """The host side is reentrant: eight threads plan different batches at
    once (ctypes releases the GIL around each call), every size equals the
    serial one, and each thread's specgen_last_error is its own call's."""
    import threading
    import paper_2606_17518_amd.binding as B
    import synth
    batches = [synth.make_fork_batch(prefix_lens=[100 + 37 * i, 50], forks_per_trace=[1 + i % 5, 2],
                                     suffix_range=(0, 90), num_q_heads=16, num_kv_heads=2,
                                     head_dim=64 if i % 2 else 128, seed=600 + i) for i in range(8)]
    structs = []
    for b in batches:
        s, keep = B.host_batch_struct(b)
        for f in ("q", "k_pool", "v_pool", "fork_off", "prefix_len", "prefix_table_off", "prefix_table",
                  "suffix_len", "suffix_table_off", "suffix_table"):
            setattr(s, f, 0x10000)   # never dereferenced: the size query reads the host mirrors only
        structs.append((s, keep))

    def size_of(s):
        n = C.c_size_t(0)
        assert L.specgen_fork_decode_attn_workspace_size(C.byref(s), C.byref(n)) == 0, L.specgen_last_error().decode()
        return n.value

    serial = [size_of(s) for s, _ in structs]
    errors = []

    def worker(i):
        try:
            s, _ = structs[i]
            bad, keep = _host_batch(num_q_heads=7)   # rejected: Hq % Hkv != 0
            for k in range(150):
                assert size_of(s) == serial[i]
                n = C.c_size_t(0)
                assert L.specgen_fork_decode_attn_workspace_size(C.byref(bad), C.byref(n)) == B.SPECGEN_ERR_INVALID_ARG
                assert "num_q_heads" in L.specgen_last_error().decode() or "Hq" in L.specgen_last_error().decode()
        except Exception as e:   # reported below: an assertion in a thread does not fail the test by itself
            errors.append((i, repr(e)))

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(8)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
