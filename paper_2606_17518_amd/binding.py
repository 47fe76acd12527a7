"""ctypes binding of libspecgen.so (include/specgen.h), argument marshalling only.

Every function here forwards to the C entry point of the same name; all the
work happens in the HIP kernels.  Device buffers are torch tensors on the
current HIP device; the stream defaults to torch's current stream.  If the
library has not been built this module raises on first use -- there is no
fallback path.
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import os
from typing import Optional, Sequence

import numpy as np
import torch

from .build import DEBUG_LIB_PATH, LIB_PATH, TIMELINE_LIB_PATH

SPECGEN_OK, SPECGEN_ERR_INVALID_ARG, SPECGEN_ERR_UNSUPPORTED, SPECGEN_ERR_WORKSPACE, SPECGEN_ERR_DEVICE = range(5)
SPECGEN_BF16, SPECGEN_FP8_E4M3, SPECGEN_FP32 = 0, 1, 2
SPECGEN_PATH_AUTO, SPECGEN_PATH_DOT, SPECGEN_PATH_MFMA = 0, 1, 2
PATHS = {"auto": SPECGEN_PATH_AUTO, "dot": SPECGEN_PATH_DOT, "mfma": SPECGEN_PATH_MFMA}

SPECGEN_PHASE_ALL, SPECGEN_PHASE_PARTIALS, SPECGEN_PHASE_MERGE = 0, 1, 2
SPECGEN_FLAG_FP8_SCORES = 1

EXPORTED = ("specgen_fork_decode_attn_workspace_size", "specgen_fork_decode_attn", "specgen_fork_decode_attn_phase",
            "specgen_fork_prefill_attn_workspace_size", "specgen_fork_prefill_attn",
            "specgen_kv_import", "specgen_kv_export", "specgen_kv_append", "specgen_lse_merge", "specgen_last_error",
            "specgen_fork_decode_attn_split", "specgen_fork_decode_attn_noalloc")


class SpecgenError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"specgen status {status}: {message}")
        self.status = status


class ForkBatchC(C.Structure):
    _fields_ = [
        ("num_traces", C.c_int32), ("num_forks", C.c_int32), ("num_q_heads", C.c_int32),
        ("num_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("block_size", C.c_int32),
        ("num_blocks", C.c_int64), ("sm_scale", C.c_float), ("kv_dtype", C.c_int32),
        ("path", C.c_int32), ("flags", C.c_int32),
        ("q", C.c_void_p), ("k_pool", C.c_void_p), ("v_pool", C.c_void_p),
        ("k_scale", C.c_void_p), ("v_scale", C.c_void_p),
        ("fork_off", C.c_void_p), ("prefix_len", C.c_void_p), ("prefix_table_off", C.c_void_p),
        ("prefix_table", C.c_void_p), ("suffix_len", C.c_void_p), ("suffix_table_off", C.c_void_p),
        ("suffix_table", C.c_void_p),
        ("fork_off_h", C.c_void_p), ("prefix_len_h", C.c_void_p), ("suffix_len_h", C.c_void_p),
        ("prefix_table_off_h", C.c_void_p), ("suffix_table_off_h", C.c_void_p),
        ("prefix_parent_h", C.c_void_p),
    ]


class SplitSegmentC(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("kind", "trace", "fork", "kv_head", "row_block", "first_row", "num_rows",
                                         "kernel", "worker", "first_token", "num_tokens")]


class KvTensorC(C.Structure):
    _fields_ = [("dst_pool", C.c_void_p), ("src_staging", C.c_void_p), ("block_bytes", C.c_int64)]


class KvExportTensorC(C.Structure):
    _fields_ = [("dst_staging", C.c_void_p), ("src_pool", C.c_void_p), ("block_bytes", C.c_int64)]


class KvAppendC(C.Structure):
    _fields_ = [
        ("num_forks", C.c_int32), ("num_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("kv_dtype", C.c_int32),
        ("num_blocks", C.c_int64),
        ("k_pool", C.c_void_p), ("v_pool", C.c_void_p), ("k_new", C.c_void_p), ("v_new", C.c_void_p),
        ("pos", C.c_void_p), ("suffix_table_off", C.c_void_p), ("suffix_table", C.c_void_p),
        ("bad_count", C.c_void_p),
    ]


_lib = None
_debug_lib = None
_timeline_lib = None


def load(path: str):
    """Loads a build of the library at `path` and declares its entry points."""
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with paper_2606_17518_amd.build.build()")
    L = C.CDLL(path)
    P = C.c_void_p
    L.specgen_fork_decode_attn_workspace_size.argtypes = [C.POINTER(ForkBatchC), C.POINTER(C.c_size_t)]
    L.specgen_fork_decode_attn_workspace_size.restype = C.c_int
    L.specgen_fork_decode_attn.argtypes = [C.POINTER(ForkBatchC), P, P, P, C.c_size_t, P]
    L.specgen_fork_decode_attn.restype = C.c_int
    L.specgen_fork_decode_attn_phase.argtypes = [C.POINTER(ForkBatchC), C.c_int32, P, P, P, C.c_size_t, P]
    L.specgen_fork_decode_attn_phase.restype = C.c_int
    L.specgen_fork_prefill_attn_workspace_size.argtypes = [C.POINTER(ForkBatchC), P, C.POINTER(C.c_size_t)]
    L.specgen_fork_prefill_attn_workspace_size.restype = C.c_int
    L.specgen_fork_prefill_attn.argtypes = [C.POINTER(ForkBatchC), P, P, P, P, C.c_size_t, P]
    L.specgen_fork_prefill_attn.restype = C.c_int
    L.specgen_kv_import.argtypes = [C.POINTER(KvTensorC), C.c_int32, P, C.c_int64, C.c_int64, P, P]
    L.specgen_kv_import.restype = C.c_int
    L.specgen_kv_export.argtypes = [C.POINTER(KvExportTensorC), C.c_int32, P, C.c_int64, C.c_int64, P, P]
    L.specgen_kv_export.restype = C.c_int
    L.specgen_kv_append.argtypes = [C.POINTER(KvAppendC), P]
    L.specgen_kv_append.restype = C.c_int
    L.specgen_lse_merge.argtypes = [P, P, C.c_int32, C.c_int64, C.c_int32, P, C.c_int32, P, P]
    L.specgen_lse_merge.restype = C.c_int
    L.specgen_fork_decode_attn_noalloc.argtypes = [C.POINTER(ForkBatchC), P, P, P]
    L.specgen_fork_decode_attn_noalloc.restype = C.c_int
    L.specgen_fork_decode_attn_split.argtypes = [C.POINTER(ForkBatchC), P, C.c_int64, C.POINTER(C.c_int64)]
    L.specgen_fork_decode_attn_split.restype = C.c_int
    L.specgen_last_error.argtypes = []
    L.specgen_last_error.restype = C.c_char_p
    return L


def lib():
    """The loaded library; raises if it was never built."""
    global _lib
    if _lib is None:
        _lib = load(LIB_PATH)
    return _lib


def debug_lib():
    """The build with SPECGEN_DEBUG_CHECKS (attention block ids checked on the
    host before every launch: a table copy and a stream synchronisation per
    call), with the same entry points."""
    global _debug_lib
    if _debug_lib is None:
        _debug_lib = load(DEBUG_LIB_PATH)
    return _debug_lib


def timeline_lib():
    """The build whose partial kernel stamps a per-workgroup timeline
    (include/specgen_timeline.h), with every entry point of the library."""
    global _timeline_lib
    if _timeline_lib is None:
        L = load(TIMELINE_LIB_PATH)
        L.specgen_timeline_shape.argtypes = [C.POINTER(C.c_int), C.POINTER(C.c_int)]
        L.specgen_timeline_read.argtypes = [C.c_void_p, C.c_void_p]
        L.specgen_timeline_clear.argtypes = []
        _timeline_lib = L
    return _timeline_lib


def _check(status: int):
    if status != SPECGEN_OK:
        raise SpecgenError(status, lib().specgen_last_error().decode())


def _dptr(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream) -> C.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    if isinstance(stream, torch.cuda.Stream):
        return C.c_void_p(stream.cuda_stream)
    return C.c_void_p(int(stream))


def _need(*bufs) -> None:
    """Each (tensor, name, bytes, dtypes or None) whose pointer goes to the
    library must be a contiguous tensor of an accepted dtype holding the bytes
    the call reads or writes, in device memory: the C ABI gets a bare pointer
    and cannot check its extent, so a short buffer would become an
    out-of-bounds access on the device.  None tensors are skipped."""
    bufs = [b for b in bufs if b[0] is not None]
    for t, what, nbytes, dtypes in bufs:
        if dtypes is not None and t.dtype not in dtypes:
            raise ValueError(f"{what}: dtype {t.dtype}, expected one of {dtypes}")
        if not t.is_contiguous():
            raise ValueError(f"{what} must be contiguous")
        if t.numel() * t.element_size() < nbytes:
            raise ValueError(f"{what} holds {t.numel() * t.element_size()} bytes; the call needs {nbytes}")
    for t, what, _, _ in bufs:
        if t.device.type != "cuda":
            raise ValueError(f"{what} must be device memory, not {t.device}")


def _need_outputs(s, rows: int, out: Optional[torch.Tensor], out_lse: Optional[torch.Tensor], workspace=None) -> None:
    """out [rows][Hq][D] bf16 and out_lse [rows][Hq] fp32 of an attention call
    (the library checks the workspace's size itself)."""
    _need((out, "out", rows * s.num_q_heads * s.head_dim * 2, (torch.bfloat16,)),
          (out_lse, "out_lse", rows * s.num_q_heads * 4, (torch.float32,)),
          (workspace, "workspace", 0, None))


@dataclasses.dataclass
class ForkBatchTensors:
    """Device tensors + host mirrors of one fork batch (see specgen_fork_batch_t)."""
    num_traces: int
    num_forks: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    num_blocks: int
    sm_scale: float
    kv_dtype: int
    q: torch.Tensor
    k_pool: torch.Tensor
    v_pool: torch.Tensor
    k_scale: Optional[torch.Tensor]
    v_scale: Optional[torch.Tensor]
    fork_off: torch.Tensor
    prefix_len: torch.Tensor
    prefix_table_off: torch.Tensor
    prefix_table: torch.Tensor
    suffix_len: torch.Tensor
    suffix_table_off: torch.Tensor
    suffix_table: torch.Tensor
    fork_off_h: np.ndarray
    prefix_len_h: np.ndarray
    suffix_len_h: np.ndarray
    prefix_table_off_h: np.ndarray
    suffix_table_off_h: np.ndarray
    path: int = SPECGEN_PATH_AUTO
    flags: int = 0                                 # SPECGEN_FLAG_FP8_SCORES or 0
    block_size: int = 16
    prefix_parent_h: Optional[np.ndarray] = None   # nested prefixes: parent trace or -1

    @staticmethod
    def from_numpy(b, device="cuda", path: str | int = "auto", flags: int = 0) -> "ForkBatchTensors":
        """Upload an object with the numpy fields of a fork batch (q, pools,
        scales, index arrays) and keep int32 host mirrors of the lengths and
        table offsets."""
        def dev(a, dt):
            return torch.from_numpy(np.ascontiguousarray(a).view(dt)).to(device)
        fp8 = b.kv_dtype != "bf16"
        kv_np = np.uint8 if fp8 else np.int16
        return ForkBatchTensors(
            num_traces=b.num_traces, num_forks=b.num_forks, num_q_heads=b.num_q_heads,
            num_kv_heads=b.num_kv_heads, head_dim=b.head_dim, num_blocks=b.num_blocks,
            sm_scale=float(b.sm_scale), kv_dtype=SPECGEN_FP8_E4M3 if fp8 else SPECGEN_BF16,
            q=dev(b.q, np.int16), k_pool=dev(b.k_pool, kv_np), v_pool=dev(b.v_pool, kv_np),
            k_scale=dev(b.k_scale, np.float32) if fp8 else None,
            v_scale=dev(b.v_scale, np.float32) if fp8 else None,
            fork_off=dev(b.fork_off, np.int32), prefix_len=dev(b.prefix_len, np.int32),
            prefix_table_off=dev(b.prefix_table_off, np.int32), prefix_table=dev(b.prefix_table, np.int32),
            suffix_len=dev(b.suffix_len, np.int32), suffix_table_off=dev(b.suffix_table_off, np.int32),
            suffix_table=dev(b.suffix_table, np.int32),
            fork_off_h=np.ascontiguousarray(b.fork_off, np.int32),
            prefix_len_h=np.ascontiguousarray(b.prefix_len, np.int32),
            suffix_len_h=np.ascontiguousarray(b.suffix_len, np.int32),
            prefix_table_off_h=np.ascontiguousarray(b.prefix_table_off, np.int32),
            suffix_table_off_h=np.ascontiguousarray(b.suffix_table_off, np.int32),
            path=PATHS[path] if isinstance(path, str) else int(path), flags=int(flags),
            prefix_parent_h=None if getattr(b, "prefix_parent", None) is None
            else np.ascontiguousarray(b.prefix_parent, np.int32))

    def c_struct(self, **overrides) -> ForkBatchC:
        s = ForkBatchC()
        s.num_traces = self.num_traces
        s.num_forks = self.num_forks
        s.num_q_heads = self.num_q_heads
        s.num_kv_heads = self.num_kv_heads
        s.head_dim = self.head_dim
        s.block_size = self.block_size
        s.num_blocks = self.num_blocks
        s.sm_scale = self.sm_scale
        s.kv_dtype = self.kv_dtype
        s.path = self.path
        s.flags = self.flags
        for name in ("q", "k_pool", "v_pool", "k_scale", "v_scale", "fork_off", "prefix_len", "prefix_table_off",
                     "prefix_table", "suffix_len", "suffix_table_off", "suffix_table"):
            t = getattr(self, name)
            setattr(s, name, None if t is None else t.data_ptr())
        for name in ("fork_off_h", "prefix_len_h", "suffix_len_h", "prefix_table_off_h", "suffix_table_off_h"):
            setattr(s, name, getattr(self, name).ctypes.data)
        s.prefix_parent_h = None if self.prefix_parent_h is None else self.prefix_parent_h.ctypes.data
        for k, v in overrides.items():
            setattr(s, k, v)
        return s


def specgen_fork_decode_attn_workspace_size(batch) -> int:
    s = batch if isinstance(batch, ForkBatchC) else batch.c_struct()
    n = C.c_size_t(0)
    _check(lib().specgen_fork_decode_attn_workspace_size(C.byref(s), C.byref(n)))
    return int(n.value)


def alloc_workspace(batch, device="cuda") -> torch.Tensor:
    n = specgen_fork_decode_attn_workspace_size(batch)
    return torch.empty(max(n, 256) // 4 + 64, dtype=torch.float32, device=device)


def specgen_fork_decode_attn(batch, out: torch.Tensor, out_lse: Optional[torch.Tensor], workspace: torch.Tensor,
                             stream=None) -> None:
    s = batch if isinstance(batch, ForkBatchC) else batch.c_struct()
    _need_outputs(s, s.num_forks, out, out_lse, workspace)
    _check(lib().specgen_fork_decode_attn(C.byref(s), _dptr(out), _dptr(out_lse), _dptr(workspace),
                                          workspace.numel() * workspace.element_size(), _stream(stream)))


SPECGEN_NOALLOC_SCRATCH_BYTES = 64 << 20   # the library's per-GPU scratch of the no-allocation call


def specgen_fork_decode_attn_noalloc(batch, out: torch.Tensor, out_lse: Optional[torch.Tensor], stream=None) -> None:
    """specgen_fork_decode_attn without a workspace: the partials live in the
    library's per-GPU scratch (calls that overlap on one GPU race)."""
    s = batch if isinstance(batch, ForkBatchC) else batch.c_struct()
    _need_outputs(s, s.num_forks, out, out_lse)
    _check(lib().specgen_fork_decode_attn_noalloc(C.byref(s), _dptr(out), _dptr(out_lse), _stream(stream)))


def specgen_fork_decode_attn_phase(batch, phase: int, out: Optional[torch.Tensor], out_lse: Optional[torch.Tensor],
                                   workspace: torch.Tensor, stream=None) -> None:
    s = batch if isinstance(batch, ForkBatchC) else batch.c_struct()
    _need_outputs(s, s.num_forks, out, out_lse, workspace)
    _check(lib().specgen_fork_decode_attn_phase(C.byref(s), int(phase), _dptr(out), _dptr(out_lse), _dptr(workspace),
                                                workspace.numel() * workspace.element_size(), _stream(stream)))


def _q_len(q_len) -> np.ndarray:
    return np.ascontiguousarray(q_len, dtype=np.int32)


def specgen_fork_prefill_attn_workspace_size(batch, q_len) -> int:
    s = batch if isinstance(batch, ForkBatchC) else batch.c_struct()
    ql = _q_len(q_len)
    n = C.c_size_t(0)
    _check(lib().specgen_fork_prefill_attn_workspace_size(C.byref(s), ql.ctypes.data_as(C.c_void_p), C.byref(n)))
    return n.value


def alloc_prefill_workspace(batch, q_len, device="cuda") -> torch.Tensor:
    n = specgen_fork_prefill_attn_workspace_size(batch, q_len)
    return torch.empty(max(1, (n + 3) // 4), dtype=torch.float32, device=device)


def specgen_fork_prefill_attn(batch, q_len, out: torch.Tensor, out_lse: Optional[torch.Tensor],
                              workspace: torch.Tensor, stream=None) -> None:
    """q_len: host int32 [N]; batch.q is [sum q_len][Hq][D]; out [sum q_len][Hq][D] bf16."""
    s = batch if isinstance(batch, ForkBatchC) else batch.c_struct()
    ql = _q_len(q_len)
    _need_outputs(s, int(ql.astype(np.int64).sum()), out, out_lse, workspace)   # one row per query
    _check(lib().specgen_fork_prefill_attn(C.byref(s), ql.ctypes.data_as(C.c_void_p), _dptr(out), _dptr(out_lse),
                                           _dptr(workspace), workspace.numel() * workspace.element_size(),
                                           _stream(stream)))


def specgen_kv_import(tensors: Sequence[tuple], dst_block_ids: torch.Tensor, num_dst_blocks: int,
                      bad_id_count: Optional[torch.Tensor] = None, stream=None) -> None:
    """tensors: sequence of (dst_pool tensor, src_staging tensor, block_bytes)."""
    arr = (KvTensorC * max(1, len(tensors)))()
    n = int(dst_block_ids.numel())
    _need((dst_block_ids, "dst_block_ids", 4 * n, (torch.int32,)),
          *[b for i, (dst, src, bb) in enumerate(tensors)
            for b in ((dst, f"tensors[{i}] dst_pool", int(num_dst_blocks) * int(bb), None),
                      (src, f"tensors[{i}] src_staging", n * int(bb), None))])
    for i, (dst, src, bb) in enumerate(tensors):
        arr[i].dst_pool = dst.data_ptr()
        arr[i].src_staging = src.data_ptr()
        arr[i].block_bytes = int(bb)
    _check(lib().specgen_kv_import(arr, len(tensors), _dptr(dst_block_ids), int(dst_block_ids.numel()),
                                   int(num_dst_blocks), _dptr(bad_id_count), _stream(stream)))


def specgen_kv_export(tensors: Sequence[tuple], src_block_ids: torch.Tensor, num_src_blocks: int,
                      bad_id_count: Optional[torch.Tensor] = None, stream=None) -> None:
    """tensors: sequence of (dst_staging tensor, src_pool tensor, block_bytes)."""
    arr = (KvExportTensorC * max(1, len(tensors)))()
    n = int(src_block_ids.numel())
    _need((src_block_ids, "src_block_ids", 4 * n, (torch.int32,)),
          *[b for i, (dst, src, bb) in enumerate(tensors)
            for b in ((dst, f"tensors[{i}] dst_staging", n * int(bb), None),
                      (src, f"tensors[{i}] src_pool", int(num_src_blocks) * int(bb), None))])
    for i, (dst, src, bb) in enumerate(tensors):
        arr[i].dst_staging = dst.data_ptr()
        arr[i].src_pool = src.data_ptr()
        arr[i].block_bytes = int(bb)
    _check(lib().specgen_kv_export(arr, len(tensors), _dptr(src_block_ids), int(src_block_ids.numel()),
                                   int(num_src_blocks), _dptr(bad_id_count), _stream(stream)))


def specgen_kv_append(k_pool: torch.Tensor, v_pool: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor,
                      pos: torch.Tensor, suffix_table_off: torch.Tensor, suffix_table: torch.Tensor,
                      num_kv_heads: int, head_dim: int, kv_dtype: int = SPECGEN_BF16, num_blocks: Optional[int] = None,
                      bad_count: Optional[torch.Tensor] = None, stream=None) -> None:
    """Pools: device tensors of 2-byte (bf16) or 1-byte (E4M3) elements; k_new,
    v_new: [N][Hkv][D] of the same element size; pos, offsets, table: int32."""
    es = 2 if kv_dtype == SPECGEN_BF16 else 1
    if num_blocks is None:
        num_blocks = k_pool.numel() * k_pool.element_size() // (num_kv_heads * 16 * head_dim * es)
    n = int(pos.numel())
    block = int(num_kv_heads) * 16 * int(head_dim) * es
    i32 = (torch.int32,)
    _need((k_pool, "k_pool", int(num_blocks) * block, None), (v_pool, "v_pool", int(num_blocks) * block, None),
          (k_new, "k_new", n * int(num_kv_heads) * int(head_dim) * es, None),
          (v_new, "v_new", n * int(num_kv_heads) * int(head_dim) * es, None),
          (pos, "pos", 4 * n, i32), (suffix_table_off, "suffix_table_off", 4 * (n + 1), i32),
          (suffix_table, "suffix_table", 0, i32), (bad_count, "bad_count", 4, i32))
    a = KvAppendC(num_forks=int(pos.numel()), num_kv_heads=int(num_kv_heads), head_dim=int(head_dim),
                  kv_dtype=int(kv_dtype), num_blocks=int(num_blocks), k_pool=k_pool.data_ptr(),
                  v_pool=v_pool.data_ptr(), k_new=k_new.data_ptr(), v_new=v_new.data_ptr(), pos=pos.data_ptr(),
                  suffix_table_off=suffix_table_off.data_ptr(), suffix_table=suffix_table.data_ptr(),
                  bad_count=None if bad_count is None else bad_count.data_ptr())
    _check(lib().specgen_kv_append(C.byref(a), _stream(stream)))


def specgen_lse_merge(o_parts: torch.Tensor, lse_parts: torch.Tensor, out: torch.Tensor,
                      out_lse: Optional[torch.Tensor] = None, stream=None) -> None:
    """o_parts [S][R][D] f32, lse_parts [S][R] f32, out [R][D] bf16 or f32."""
    S, R, D = o_parts.shape
    _need((o_parts, "o_parts", S * R * D * 4, (torch.float32,)), (lse_parts, "lse_parts", S * R * 4, (torch.float32,)),
          (out, "out", R * D * out.element_size(), (torch.bfloat16, torch.float32)),
          (out_lse, "out_lse", R * 4, (torch.float32,)))
    dt = SPECGEN_BF16 if out.dtype == torch.bfloat16 else SPECGEN_FP32
    _check(lib().specgen_lse_merge(_dptr(o_parts), _dptr(lse_parts), S, R, D, _dptr(out), dt, _dptr(out_lse),
                                   _stream(stream)))


def host_batch_struct(b, path: str | int = "auto"):
    """A ForkBatchC for the host-only queries from an object with a fork
    batch's numpy fields: the host mirrors are set, the device pointers NULL.
    Returns (struct, arrays the struct points into, to be kept alive)."""
    keep = [np.ascontiguousarray(a, np.int32) for a in
            (b.fork_off, b.prefix_len, b.suffix_len, b.prefix_table_off, b.suffix_table_off)]
    s = ForkBatchC()
    s.num_traces, s.num_forks, s.num_q_heads, s.num_kv_heads = b.num_traces, b.num_forks, b.num_q_heads, b.num_kv_heads
    s.head_dim, s.block_size, s.num_blocks, s.sm_scale = b.head_dim, 16, b.num_blocks, float(b.sm_scale)
    s.kv_dtype = SPECGEN_BF16 if b.kv_dtype == "bf16" else SPECGEN_FP8_E4M3
    s.path = PATHS[path] if isinstance(path, str) else int(path)
    s.flags = 0
    s.fork_off_h, s.prefix_len_h, s.suffix_len_h, s.prefix_table_off_h, s.suffix_table_off_h = \
        (a.ctypes.data for a in keep)
    if getattr(b, "prefix_parent", None) is not None:
        keep.append(np.ascontiguousarray(b.prefix_parent, np.int32))
        s.prefix_parent_h = keep[-1].ctypes.data
    return s, keep


def specgen_fork_decode_attn_split(batch, path: str | int = "auto") -> dict:
    """The key-axis split of a batch (host only).  `batch` is a ForkBatchC, a
    ForkBatchTensors, or an object with a fork batch's numpy fields.  Returns a
    dict of int32 arrays, one entry per segment, keyed by the fields of
    specgen_split_segment_t."""
    keep = None
    if isinstance(batch, ForkBatchC):
        s = batch
    elif isinstance(batch, ForkBatchTensors):
        s = batch.c_struct()
    else:
        s, keep = host_batch_struct(batch, path)
    n = C.c_int64(0)
    _check(lib().specgen_fork_decode_attn_split(C.byref(s), None, 0, C.byref(n)))
    arr = (SplitSegmentC * max(1, n.value))()
    _check(lib().specgen_fork_decode_attn_split(C.byref(s), arr, n.value, C.byref(n)))
    del keep
    names = [f for f, _ in SplitSegmentC._fields_]
    raw = np.frombuffer(arr, dtype=np.int32, count=n.value * len(names)).reshape(n.value, len(names))
    return {name: raw[:, i].copy() for i, name in enumerate(names)}
