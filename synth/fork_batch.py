"""Seeded synthetic inputs for fork-decode attention and KV-block import.

This module only draws and places data: lengths, block tables, bf16 / OCP E4M3
tensors, NaN poisoning of slots no valid token occupies.  It holds none of the
attention, merge or import arithmetic, so both the oracle and the HIP path can
consume the very same bytes.

Draw order (numpy PCG64, one generator per batch):
  1. lengths (prefix lengths if drawn, then suffix lengths, fork by fork);
  2. one random permutation of the pool's block ids; prefix tables take the
     first ids trace by trace, then suffix tables fork by fork;
  3. q ~ N(0, 1), rounded to bf16 (round-to-nearest-even);
  4. the per-kv-head key bias (only when key_bias_std > 0), then K for every
     valid token (all prefixes, then all suffixes, in logical order), then V;
     values N(0, 1) (plus the bias for K) rounded to bf16, or quantised to
     E4M3 with one fp32 scale per physical block = amax / 448 (1 if amax = 0);
  5. every pool slot that holds no valid token is set to NaN (bf16 0x7FC0,
     E4M3 0x7F), as is the scale of every unused block.

Pool layout (one block of 16 tokens is contiguous, each kv head's slice of a
block is contiguous inside it):
  K pool [num_blocks][Hkv][16][D]  -- token rows of D elements;
  V pool [num_blocks][Hkv][D][16]  -- transposed: rows of 16 tokens per dim.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence

import numpy as np
import torch

BLOCK = 16
BF16_NAN = np.uint16(0x7FC0)
E4M3_NAN = np.uint8(0x7F)
E4M3_MAX = 448.0


@dataclasses.dataclass
class ForkBatch:
    num_traces: int
    num_forks: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    num_blocks: int
    sm_scale: float
    kv_dtype: str                       # "bf16" | "fp8_e4m3"
    q: np.ndarray                       # [N][Hq][D] uint16 (bf16 bits)
    k_pool: np.ndarray                  # [NB][Hkv][bs][D] uint16 bits or uint8 codes
    v_pool: np.ndarray                  # [NB][Hkv][D][bs]
    k_scale: Optional[np.ndarray]       # [NB] float32 (E4M3 only)
    v_scale: Optional[np.ndarray]
    fork_off: np.ndarray                # [T+1] int32
    prefix_len: np.ndarray              # [T]
    prefix_table_off: np.ndarray        # [T+1]
    prefix_table: np.ndarray
    suffix_len: np.ndarray              # [N]
    suffix_table_off: np.ndarray        # [N+1]
    suffix_table: np.ndarray
    seed: int = 0
    name: str = ""
    # logical (pre-paging) K/V per segment, kept only on request: list of
    # [len][Hkv][D] arrays, prefixes of traces 0..T-1 then suffixes of forks 0..N-1
    k_logical: Optional[list] = None
    v_logical: Optional[list] = None
    # E4M3 only: per-token scale [len] of the block each logical token sits in
    k_logical_scale: Optional[list] = None
    v_logical_scale: Optional[list] = None
    # nested prefixes: parent trace of each trace (-1 for a root), or None
    prefix_parent: Optional[np.ndarray] = None
    # multi-token prefill: queries per fork (q is then [sum q_len][Hq][D]), or None
    q_len: Optional[np.ndarray] = None

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    def trace_of_fork(self, f: int) -> int:
        return int(np.searchsorted(self.fork_off, f, side="right") - 1)

    def prefix_chain(self, t: int) -> list:
        """Traces whose prefix tokens precede a fork of trace t, root first."""
        chain = []
        while t >= 0:
            chain.append(t)
            t = -1 if self.prefix_parent is None else int(self.prefix_parent[t])
        return chain[::-1]

    def keys_of_fork(self, f: int) -> int:
        return sum(int(self.prefix_len[c]) for c in self.prefix_chain(self.trace_of_fork(f))) + int(self.suffix_len[f])

    def kv_elem_bytes(self) -> int:
        return 2 if self.kv_dtype == "bf16" else 1

    def block_bytes(self) -> int:
        return self.block_size * self.num_kv_heads * self.head_dim * self.kv_elem_bytes()

    def algorithmic_bytes(self) -> int:
        """HBM bytes one decode step must move at minimum: every valid prefix
        token's K and V once per kv head, every suffix token's K and V once,
        the E4M3 block scales actually used, q in, out (bf16) and lse (fp32)
        out, and the index arrays."""
        e = self.kv_elem_bytes()
        per_tok = 2 * self.num_kv_heads * self.head_dim * e
        kv = per_tok * (int(self.prefix_len.sum()) + int(self.suffix_len.sum()))
        scales = 0
        if self.kv_dtype != "bf16":
            used = len(self.prefix_table) + len(self.suffix_table)
            scales = 2 * 4 * used
        qo = self.num_forks * self.num_q_heads * (self.head_dim * 2 * 2 + 4)
        idx = 4 * (len(self.fork_off) + len(self.prefix_len) + len(self.prefix_table_off)
                   + len(self.prefix_table) + len(self.suffix_len) + len(self.suffix_table_off)
                   + len(self.suffix_table))
        return kv + scales + qo + idx

    def flops(self) -> int:
        """Multiply-adds x2 of QK^T and PV over every (fork, q head) row."""
        toks = sum(self.keys_of_fork(f) for f in range(self.num_forks))
        return 4 * self.head_dim * self.num_q_heads * toks


def _to_bf16_bits(x: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _to_e4m3_codes(x: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def make_fork_batch(*, prefix_lens: Sequence[int] | None = None,
                    prefix_range: tuple | None = None, num_traces: int = 1,
                    forks_per_trace: int | Sequence[int] = 1,
                    suffix_range: tuple = (0, 0), suffix_lens: Sequence[int] | None = None,
                    num_q_heads: int = 8, num_kv_heads: int = 2, head_dim: int = 64,
                    kv_dtype: str = "bf16", key_bias_std: float = 0.0,
                    num_blocks: int | None = None, extra_blocks: int | None = None,
                    sm_scale: float | None = None, seed: int = 0, name: str = "",
                    keep_logical: bool = False, identity_table: bool = False,
                    prefix_parent: Sequence[int] | None = None) -> ForkBatch:
    """Draw one fork batch.  Integer ranges are inclusive of both ends.
    ``prefix_parent`` makes the traces' prefixes nested: trace t's own prefix
    tokens follow the whole prefix of trace prefix_parent[t] (-1: a root); the
    traces must be listed in depth-first order."""
    rng = np.random.default_rng(seed)
    bs = BLOCK
    # 1. lengths
    if prefix_lens is not None:
        P = np.asarray(prefix_lens, dtype=np.int64)
        T = len(P)
    else:
        T = num_traces
        lo, hi = prefix_range
        P = rng.integers(lo, hi + 1, size=T).astype(np.int64)
    if isinstance(forks_per_trace, (int, np.integer)):
        F = np.full(T, int(forks_per_trace), dtype=np.int64)
    else:
        F = np.asarray(forks_per_trace, dtype=np.int64)
    N = int(F.sum())
    if suffix_lens is not None:
        S = np.asarray(suffix_lens, dtype=np.int64)
        assert len(S) == N
    else:
        lo, hi = suffix_range
        S = rng.integers(lo, hi + 1, size=N).astype(np.int64)
    fork_off = np.zeros(T + 1, np.int64)
    fork_off[1:] = np.cumsum(F)

    # 2. block tables from one permutation of the pool
    nbp = [(int(p) + bs - 1) // bs for p in P]
    nbs = [(int(s) + bs - 1) // bs for s in S]
    needed = sum(nbp) + sum(nbs)
    if num_blocks is None:
        num_blocks = needed + (needed if extra_blocks is None else extra_blocks)
    assert num_blocks >= needed, "pool too small"
    perm = np.arange(num_blocks) if identity_table else rng.permutation(num_blocks)
    pos = 0
    prefix_table_off = np.zeros(T + 1, np.int64)
    suffix_table_off = np.zeros(N + 1, np.int64)
    for t in range(T):
        prefix_table_off[t + 1] = prefix_table_off[t] + nbp[t]
    prefix_table = perm[pos:pos + sum(nbp)].copy()
    pos += sum(nbp)
    for f in range(N):
        suffix_table_off[f + 1] = suffix_table_off[f] + nbs[f]
    suffix_table = perm[pos:pos + sum(nbs)].copy()

    Hq, Hkv, D = num_q_heads, num_kv_heads, head_dim
    assert Hq % Hkv == 0
    # 3. q
    q = _to_bf16_bits(rng.standard_normal((N, Hq, D), dtype=np.float32))

    # 4. K then V for every valid token, segment by segment in logical order
    segs = [(prefix_table[prefix_table_off[t]:prefix_table_off[t + 1]], int(P[t])) for t in range(T)]
    segs += [(suffix_table[suffix_table_off[f]:suffix_table_off[f + 1]], int(S[f])) for f in range(N)]
    bias = None
    if key_bias_std > 0:
        bias = rng.normal(0.0, key_bias_std, size=(Hkv, D)).astype(np.float32)
    fp8 = kv_dtype != "bf16"
    assert kv_dtype in ("bf16", "fp8_e4m3")
    el_dt = np.uint8 if fp8 else np.uint16
    nan = E4M3_NAN if fp8 else BF16_NAN
    pools, scales, logical, logical_sc = [], [], [], []
    for which in ("k", "v"):
        # pools are built token-major ([NB][bs][Hkv][D]) and laid out at the end
        pool = np.full((num_blocks, bs, Hkv, D), nan, dtype=el_dt)
        scale = np.full(num_blocks, np.nan, dtype=np.float32) if fp8 else None
        seg_logical = [] if keep_logical else None
        seg_sc = [] if keep_logical else None
        for blocks, n in segs:
            if n == 0:
                if keep_logical:
                    seg_logical.append(np.zeros((0, Hkv, D), el_dt))
                    seg_sc.append(np.zeros((0,), np.float32))
                continue
            x = rng.standard_normal((n, Hkv, D), dtype=np.float32)
            if which == "k" and bias is not None:
                x += bias[None, :, :]
            nb = len(blocks)
            padded = np.zeros((nb * bs, Hkv, D), np.float32)
            padded[:n] = x
            padded = padded.reshape(nb, bs, Hkv, D)
            if fp8:
                amax = np.abs(padded).reshape(nb, -1).max(axis=1)
                sc = np.where(amax > 0, amax / np.float32(E4M3_MAX), np.float32(1.0)).astype(np.float32)
                codes = _to_e4m3_codes(padded / sc[:, None, None, None])
                scale[blocks] = sc
                enc = codes
            else:
                enc = _to_bf16_bits(padded)
            flat = enc.reshape(nb * bs, Hkv, D)
            # only valid slots are written; the rest of the pool stays NaN
            full, rem = divmod(n, bs)
            if full:
                pool[blocks[:full]] = enc[:full]
            if rem:
                pool[blocks[full], :rem] = enc[full, :rem]
            if keep_logical:
                seg_logical.append(flat[:n].copy())
                seg_sc.append(np.repeat(scale[blocks], bs)[:n].copy() if fp8 else np.ones(n, np.float32))
        # K: [NB][Hkv][bs][D]; V: [NB][Hkv][D][bs]
        axes = (0, 2, 1, 3) if which == "k" else (0, 2, 3, 1)
        pools.append(np.ascontiguousarray(pool.transpose(axes)))
        scales.append(scale)
        logical.append(seg_logical)
        logical_sc.append(seg_sc)

    if sm_scale is None:
        sm_scale = 1.0 / math.sqrt(D)
    i32 = lambda a: np.ascontiguousarray(a, dtype=np.int32)
    return ForkBatch(
        num_traces=T, num_forks=N, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D,
        block_size=bs, num_blocks=int(num_blocks), sm_scale=float(sm_scale), kv_dtype=kv_dtype,
        q=q, k_pool=pools[0], v_pool=pools[1], k_scale=scales[0], v_scale=scales[1],
        fork_off=i32(fork_off), prefix_len=i32(P), prefix_table_off=i32(prefix_table_off),
        prefix_table=i32(prefix_table), suffix_len=i32(S), suffix_table_off=i32(suffix_table_off),
        suffix_table=i32(suffix_table), seed=seed, name=name,
        prefix_parent=None if prefix_parent is None else i32(prefix_parent),
        k_logical=logical[0] if keep_logical else None,
        v_logical=logical[1] if keep_logical else None,
        k_logical_scale=logical_sc[0] if keep_logical else None,
        v_logical_scale=logical_sc[1] if keep_logical else None)


# ---- import workloads --------------------------------------------------------

@dataclasses.dataclass
class ImportCase:
    num_tensors: int
    block_bytes: int
    n: int                      # staging blocks
    num_dst_blocks: int         # pool capacity
    staging: list               # num_tensors x uint8 [n * block_bytes]
    pool: list                  # num_tensors x uint8 [num_dst_blocks * block_bytes] (initial)
    dst_ids: np.ndarray         # int32 [n]

    def algorithmic_bytes(self) -> int:
        valid = int(((self.dst_ids >= 0) & (self.dst_ids < self.num_dst_blocks)).sum())
        return self.num_tensors * 2 * valid * self.block_bytes + 4 * self.n


SENTINEL = 0xA5


def make_import_case(*, n: int, num_dst_blocks: int, block_bytes: int, num_tensors: int = 2,
                     seed: int = 0, bad_ids: Sequence[int] = ()) -> ImportCase:
    """Random staging bytes, a sentinel-filled pool, and destination ids drawn as
    the first n entries of a random permutation of the pool (so all distinct).
    ``bad_ids`` lists staging indices whose id is replaced by an out-of-range
    value (alternately -1 and num_dst_blocks + index)."""
    rng = np.random.default_rng(seed)
    dst = rng.permutation(num_dst_blocks)[:n].astype(np.int32)
    for k, i in enumerate(bad_ids):
        dst[i] = -1 if k % 2 == 0 else num_dst_blocks + i
    staging = [rng.integers(0, 256, size=n * block_bytes, dtype=np.uint8) for _ in range(num_tensors)]
    pool = [np.full(num_dst_blocks * block_bytes, SENTINEL, dtype=np.uint8) for _ in range(num_tensors)]
    return ImportCase(num_tensors, block_bytes, n, num_dst_blocks, staging, pool, dst)


def prefix_import_from_batch(batch: ForkBatch, trace: int = 0):
    """Staging copies of one trace's prefix blocks (the state a remote cache
    holds) and the pool ids they restore into.  Returns (k_staging, v_staging,
    dst_ids, k_scale_staging, v_scale_staging); the scale entries are None for
    bf16.  The staging arrays are [n][block] views of the pool bytes."""
    ids = batch.prefix_table[batch.prefix_table_off[trace]:batch.prefix_table_off[trace + 1]].copy()
    ks = np.ascontiguousarray(batch.k_pool[ids])
    vs = np.ascontiguousarray(batch.v_pool[ids])
    kss = vss = None
    if batch.kv_dtype != "bf16":
        kss = np.ascontiguousarray(batch.k_scale[ids])
        vss = np.ascontiguousarray(batch.v_scale[ids])
    return ks, vs, ids.astype(np.int32), kss, vss


# ---- per-step append workloads -------------------------------------------------

@dataclasses.dataclass
class AppendCase:
    num_kv_heads: int
    head_dim: int
    elem_dtype: type            # np.uint16 (bf16 bits) or np.uint8 (E4M3 codes)
    k_new: np.ndarray           # [N][Hkv][D]
    v_new: np.ndarray
    pos: np.ndarray             # int32 [N], the suffix slot each new token takes
    suffix_table_off: np.ndarray  # int32 [N+1]
    suffix_table: np.ndarray      # int32
    fresh_blocks: np.ndarray      # int32, the pool blocks opened by this step

    @property
    def num_forks(self) -> int:
        return int(self.pos.size)

    def algorithmic_bytes(self) -> int:
        """New K and V read once and written once, positions, offsets and one
        table entry per fork."""
        e = np.dtype(self.elem_dtype).itemsize
        return 2 * 2 * self.k_new.size * e + 4 * (2 * self.num_forks + 1) + 4 * self.num_forks


def make_append_case(batch: ForkBatch, seed: int = 0, bad_forks: Sequence[int] = ()) -> AppendCase:
    """The next decode token of every fork of ``batch``: random K/V elements,
    position = the current suffix length, and the batch's suffix tables with a
    fresh block (a pool block no table uses) appended for every fork whose
    suffix length is a multiple of 16.  ``bad_forks`` get a position past
    their table (alternately) or a table entry outside the pool."""
    rng = np.random.default_rng(seed)
    N, Hkv, D = batch.num_forks, batch.num_kv_heads, batch.head_dim
    fp8 = batch.kv_dtype != "bf16"
    el = np.uint8 if fp8 else np.uint16
    if fp8:
        k_new = _to_e4m3_codes(rng.uniform(-448, 448, size=(N, Hkv, D)).astype(np.float32))
        v_new = _to_e4m3_codes(rng.uniform(-448, 448, size=(N, Hkv, D)).astype(np.float32))
    else:
        k_new = _to_bf16_bits(rng.standard_normal((N, Hkv, D), dtype=np.float32))
        v_new = _to_bf16_bits(rng.standard_normal((N, Hkv, D), dtype=np.float32))
    used = np.zeros(batch.num_blocks, bool)
    used[batch.prefix_table] = True
    used[batch.suffix_table] = True
    free = rng.permutation(np.flatnonzero(~used))
    pos = batch.suffix_len.astype(np.int64).copy()
    off = np.zeros(N + 1, np.int64)
    table = []
    nfree = 0
    for f in range(N):
        ids = list(batch.suffix_table[batch.suffix_table_off[f]:batch.suffix_table_off[f + 1]])
        if pos[f] % BLOCK == 0:
            assert nfree < free.size, "pool has no free block for a fresh suffix block"
            ids.append(int(free[nfree]))
            nfree += 1
        table += ids
        off[f + 1] = off[f] + len(ids)
    table = np.asarray(table, np.int64)
    for k, f in enumerate(bad_forks):
        if k % 2 == 0:
            pos[f] = (off[f + 1] - off[f]) * BLOCK        # no table entry for this position
        else:
            table[off[f] + pos[f] // BLOCK] = batch.num_blocks + f
    i32 = lambda a: np.ascontiguousarray(a, dtype=np.int32)
    return AppendCase(Hkv, D, el, k_new, v_new, i32(pos), i32(off), i32(table), i32(free[:nfree]))


# ---- multi-token prefill workloads -----------------------------------------------

def with_prefill_queries(batch: ForkBatch, q_len: Sequence[int], seed: int = 0) -> ForkBatch:
    """A copy of ``batch`` whose forks each carry q_len[f] queries (their last
    q_len[f] suffix tokens, which the suffix already holds): q becomes
    [sum q_len][Hq][D] bf16 drawn from N(0, 1), and ``q_len`` is attached."""
    ql = np.ascontiguousarray(q_len, dtype=np.int32)
    assert ql.size == batch.num_forks and np.all(ql >= 1) and np.all(ql <= batch.suffix_len)
    rng = np.random.default_rng(seed)
    out = dataclasses.replace(batch)
    out.q = _to_bf16_bits(rng.standard_normal((int(ql.sum()), batch.num_q_heads, batch.head_dim), dtype=np.float32))
    out.q_len = ql
    return out


# ---- peaked queries -------------------------------------------------------------

def logical_key(batch: ForkBatch, f: int, j: int, i: int) -> np.ndarray:
    """The value of key i (0-based, logical order: the prefix chain of fork
    f's trace, root first, then f's suffix) of kv head j as float32: the bf16
    bits widened, or the E4M3 code decoded and multiplied by its block scale.
    This reads back the generator's own placement."""
    bs = batch.block_size
    blk = slot = None
    for t in batch.prefix_chain(batch.trace_of_fork(f)):
        n = int(batch.prefix_len[t])
        if i < n:
            blk = int(batch.prefix_table[batch.prefix_table_off[t] + i // bs])
            slot = i % bs
            break
        i -= n
    if blk is None:
        assert 0 <= i < int(batch.suffix_len[f]), "key index past the fork's keys"
        blk = int(batch.suffix_table[batch.suffix_table_off[f] + i // bs])
        slot = i % bs
    row = batch.k_pool[blk, j, slot]
    if batch.kv_dtype == "bf16":
        return (row.astype(np.uint32) << 16).view(np.float32)
    dec = torch.from_numpy(np.ascontiguousarray(row)).view(torch.float8_e4m3fn).to(torch.float32).numpy()
    return dec * batch.k_scale[blk]


def with_peaked_queries(batch: ForkBatch, key_index: np.ndarray, weight: np.ndarray, q_scale: float) -> ForkBatch:
    """A copy of ``batch`` whose queries make attention peaked:
    q[f][h] = q_scale * q0[f][h] + weight[f][h] * k, rounded to bf16, where q0
    is the batch's own query and k the logical key key_index[f][h] of the
    fork's kv head for h (no key where key_index < 0).  With N(0, 1) keys and
    scale 1/sqrt(D), the scores of a row spread with standard deviation about
    sqrt(q_scale^2 + weight^2) and the chosen key scores about weight * |k|^2
    / sqrt(D) above zero, so it dominates its row for weight >= 2."""
    N, Hq, D, g = batch.num_forks, batch.num_q_heads, batch.head_dim, batch.group
    q0 = (batch.q.astype(np.uint32) << 16).view(np.float32).reshape(N, Hq, D)
    q = q_scale * q0
    for f in range(N):
        for h in range(Hq):
            if key_index[f, h] >= 0:
                q[f, h] += np.float32(weight[f, h]) * logical_key(batch, f, h // g, int(key_index[f, h]))
    out = dataclasses.replace(batch)
    out.q = _to_bf16_bits(q)
    return out
