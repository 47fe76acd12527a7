"""fp64 CPU oracle for SpecGen's fork-decode attention, LSE merge, KV import/export and append.

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg are the only users.  The product library
(``paper_2606_17518_amd``) never imports this package, and this package
imports nothing from it.

The computation lives in ``specgen_oracle.c`` (plain C, fp64, OpenMP over
output rows); this module compiles it with gcc on first use and marshals
numpy arrays through ctypes.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "specgen_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libspecgen_oracle.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (fp64, no FMA contraction, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
               "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class RefBatch(C.Structure):
    _fields_ = [
        ("num_traces", C.c_int32), ("num_forks", C.c_int32),
        ("num_q_heads", C.c_int32), ("num_kv_heads", C.c_int32),
        ("head_dim", C.c_int32), ("block_size", C.c_int32),
        ("num_blocks", C.c_int64),
        ("sm_scale", C.c_double),
        ("kv_dtype", C.c_int32), ("pad_", C.c_int32),
        ("q", C.c_void_p),
        ("k_pool", C.c_void_p), ("v_pool", C.c_void_p),
        ("k_scale", C.c_void_p), ("v_scale", C.c_void_p),
        ("fork_off", C.c_void_p), ("prefix_len", C.c_void_p),
        ("prefix_table_off", C.c_void_p), ("prefix_table", C.c_void_p),
        ("suffix_len", C.c_void_p), ("suffix_table_off", C.c_void_p),
        ("suffix_table", C.c_void_p), ("prefix_parent", C.c_void_p),
    ]


def _load():
    global _lib
    with _lock:
        if _lib is None:
            lib = C.CDLL(build())
            P = C.c_void_p
            lib.specgen_ref_attend_dense.argtypes = [P, P, P, C.c_int64, C.c_int32, C.c_double, P, P]
            lib.specgen_ref_attend_dense.restype = None
            lib.specgen_ref_fork_decode_attn.argtypes = [C.POINTER(RefBatch), P, C.c_int64, P, P, C.c_int32]
            lib.specgen_ref_fork_decode_attn.restype = C.c_int
            lib.specgen_ref_fork_prefill_attn.argtypes = [C.POINTER(RefBatch), P, P, C.c_int64, P, P, C.c_int32]
            lib.specgen_ref_fork_prefill_attn.restype = C.c_int
            lib.specgen_ref_lse_merge.argtypes = [P, P, C.c_int32, C.c_int64, C.c_int32, P, P]
            lib.specgen_ref_lse_merge.restype = None
            lib.specgen_ref_kv_import.argtypes = [P, P, C.c_int64, P, C.c_int64, C.c_int64]
            lib.specgen_ref_kv_import.restype = C.c_int64
            lib.specgen_ref_kv_export.argtypes = [P, P, C.c_int64, P, C.c_int64, C.c_int64]
            lib.specgen_ref_kv_export.restype = C.c_int64
            lib.specgen_ref_kv_append.argtypes = [P, P, P, P, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                                  P, P, P, C.c_int64]
            lib.specgen_ref_kv_append.restype = C.c_int64
            lib.specgen_ref_decode_bf16.argtypes = [P, C.c_int64, P]
            lib.specgen_ref_decode_e4m3.argtypes = [P, C.c_int64, P]
            lib.specgen_ref_max_threads.restype = C.c_int32
            _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def max_threads() -> int:
    return int(_load().specgen_ref_max_threads())


def bf16_to_f64(bits) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns (uint16) to float64."""
    src = _c(bits, np.uint16)
    out = np.empty(src.shape, np.float64)
    _load().specgen_ref_decode_bf16(_ptr(src), src.size, _ptr(out))
    return out


def e4m3_to_f64(codes) -> np.ndarray:
    """OCP E4M3 (FN) decode of uint8 codes to float64."""
    src = _c(codes, np.uint8)
    out = np.empty(src.shape, np.float64)
    _load().specgen_ref_decode_e4m3(_ptr(src), src.size, _ptr(out))
    return out


def attend_dense(q, K, V, sm_scale: float):
    """Single-query softmax attention by definition: q [D], K/V [n][D] float64.
    Returns (o [D], lse) with lse in natural log."""
    q = _c(q, np.float64)
    K = _c(K, np.float64)
    V = _c(V, np.float64)
    D = q.shape[0]
    n = K.shape[0] if K.ndim == 2 else 0
    o = np.empty(D, np.float64)
    lse = np.empty(1, np.float64)
    _load().specgen_ref_attend_dense(_ptr(q), _ptr(K), _ptr(V), n, D, float(sm_scale), _ptr(o), _ptr(lse))
    return o, float(lse[0])


def _ref_batch(b, keep):
    def hold(a, dt):
        a = _c(a, dt)
        keep.append(a)
        return _ptr(a)

    rb = RefBatch()
    rb.num_traces = b.num_traces
    rb.num_forks = b.num_forks
    rb.num_q_heads = b.num_q_heads
    rb.num_kv_heads = b.num_kv_heads
    rb.head_dim = b.head_dim
    rb.block_size = b.block_size
    rb.num_blocks = b.num_blocks
    rb.sm_scale = float(b.sm_scale)
    rb.kv_dtype = 0 if b.kv_dtype == "bf16" else 1
    rb.q = hold(b.q, np.uint16)
    kv_np = np.uint16 if b.kv_dtype == "bf16" else np.uint8
    rb.k_pool = hold(b.k_pool, kv_np)
    rb.v_pool = hold(b.v_pool, kv_np)
    if b.kv_dtype != "bf16":
        rb.k_scale = hold(b.k_scale, np.float32)
        rb.v_scale = hold(b.v_scale, np.float32)
    rb.fork_off = hold(b.fork_off, np.int32)
    rb.prefix_len = hold(b.prefix_len, np.int32)
    rb.prefix_table_off = hold(b.prefix_table_off, np.int32)
    rb.prefix_table = hold(b.prefix_table, np.int32)
    rb.suffix_len = hold(b.suffix_len, np.int32)
    rb.suffix_table_off = hold(b.suffix_table_off, np.int32)
    rb.suffix_table = hold(b.suffix_table, np.int32)
    parent = getattr(b, "prefix_parent", None)
    rb.prefix_parent = None if parent is None else hold(parent, np.int32)
    return rb


def _rows_out(rows, n_all, D, keep):
    if rows is None:
        return None, 0, np.empty((n_all, D), np.float64), np.empty((n_all,), np.float64)
    rows_a = _c(rows, np.int32).reshape(-1, 2)
    keep.append(rows_a)
    n = rows_a.shape[0]
    return _ptr(rows_a), n, np.empty((n, D), np.float64), np.empty((n,), np.float64)


def fork_decode_attn(batch, rows=None, nthreads: int = 0):
    """Oracle fork-decode attention for a ``synth`` ForkBatch (numpy arrays).

    rows: optional int array [n][2] of (fork, q head) pairs; default all rows.
    Returns (out, lse): [N][Hq][D] and [N][Hq] (or [n][D], [n]) float64.
    """
    keep = []
    rb = _ref_batch(batch, keep)
    N, Hq, D = batch.num_forks, batch.num_q_heads, batch.head_dim
    rows_p, n, out, lse = _rows_out(rows, N * Hq, D, keep)
    rc = _load().specgen_ref_fork_decode_attn(C.byref(rb), rows_p, n, _ptr(out), _ptr(lse), int(nthreads))
    if rc != 0:
        raise ValueError("oracle: malformed fork batch")
    if rows is None:
        return out.reshape(N, Hq, D), lse.reshape(N, Hq)
    return out, lse


def fork_prefill_attn(batch, q_len, rows=None, nthreads: int = 0):
    """Oracle multi-token prefill: fork f's last q_len[f] suffix tokens are
    queries (batch.q is [sum q_len][Hq][D]), causal inside the suffix.

    rows: optional int array [n][2] of (query index, q head) pairs.
    Returns (out, lse): [sum q_len][Hq][D] and [sum q_len][Hq] (or [n][D], [n])."""
    keep = []
    rb = _ref_batch(batch, keep)
    ql = _c(q_len, np.int32)
    keep.append(ql)
    nq, Hq, D = int(ql.sum()), batch.num_q_heads, batch.head_dim
    rows_p, n, out, lse = _rows_out(rows, nq * Hq, D, keep)
    rc = _load().specgen_ref_fork_prefill_attn(C.byref(rb), _ptr(ql), rows_p, n, _ptr(out), _ptr(lse),
                                               int(nthreads))
    if rc != 0:
        raise ValueError("oracle: malformed prefill batch")
    if rows is None:
        return out.reshape(nq, Hq, D), lse.reshape(nq, Hq)
    return out, lse


def lse_merge(o_parts, lse_parts):
    """Merge partial (o, lse): o_parts [S][R][D] f32, lse_parts [S][R] f32.
    Returns (out [R][D], lse [R]) float64."""
    o = _c(o_parts, np.float32)
    l = _c(lse_parts, np.float32)
    S, R, D = o.shape
    out = np.empty((R, D), np.float64)
    lse = np.empty((R,), np.float64)
    _load().specgen_ref_lse_merge(_ptr(o), _ptr(l), S, R, D, _ptr(out), _ptr(lse))
    return out, lse


def kv_import(dst_pool: np.ndarray, src: np.ndarray, block_bytes: int, dst_ids, num_dst_blocks: int) -> int:
    """Naive block copy, in place on ``dst_pool`` (uint8, contiguous).
    Returns the number of skipped (out-of-range) ids."""
    assert dst_pool.dtype == np.uint8 and dst_pool.flags.c_contiguous
    s = _c(src, np.uint8)
    ids = _c(dst_ids, np.int32)
    return int(_load().specgen_ref_kv_import(_ptr(dst_pool), _ptr(s), int(block_bytes), _ptr(ids),
                                             ids.size, int(num_dst_blocks)))


def kv_export(staging: np.ndarray, pool: np.ndarray, block_bytes: int, src_ids, num_src_blocks: int) -> int:
    """Naive block gather, in place on ``staging`` (uint8, contiguous): staging
    block i receives pool block src_ids[i].  Returns the number of skipped ids."""
    assert staging.dtype == np.uint8 and staging.flags.c_contiguous
    p = _c(pool, np.uint8)
    ids = _c(src_ids, np.int32)
    return int(_load().specgen_ref_kv_export(_ptr(staging), _ptr(p), int(block_bytes), _ptr(ids),
                                             ids.size, int(num_src_blocks)))


def kv_append(k_pool: np.ndarray, v_pool: np.ndarray, k_new, v_new, pos, suffix_table_off, suffix_table,
              num_kv_heads: int, head_dim: int) -> int:
    """Write each fork's new token into its suffix blocks, in place on the pools.

    Pools are contiguous arrays of 1- or 2-byte elements (uint8 codes or uint16
    bf16 bits) holding num_blocks * Hkv * 16 * D elements; k_new / v_new are
    [N][Hkv][D] of the same element type.  Returns the number of skipped forks."""
    assert k_pool.dtype == v_pool.dtype and k_pool.flags.c_contiguous and v_pool.flags.c_contiguous
    es = k_pool.dtype.itemsize
    assert es in (1, 2)
    kn = _c(k_new, k_pool.dtype)
    vn = _c(v_new, k_pool.dtype)
    pos = _c(pos, np.int32)
    off = _c(suffix_table_off, np.int32)
    tab = _c(suffix_table if suffix_table is not None and np.size(suffix_table) else np.zeros(1, np.int32), np.int32)
    n = pos.size
    assert kn.size == vn.size == n * num_kv_heads * head_dim and off.size == n + 1
    nblocks = k_pool.size // (num_kv_heads * 16 * head_dim)
    return int(_load().specgen_ref_kv_append(_ptr(k_pool), _ptr(v_pool), _ptr(kn), _ptr(vn), es, n,
                                             int(num_kv_heads), int(head_dim), _ptr(pos), _ptr(off), _ptr(tab),
                                             nblocks))
