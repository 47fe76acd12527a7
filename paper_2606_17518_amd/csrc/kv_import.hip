// kv_import.hip -- block-table-driven moves of whole KV blocks between the
// paged pool and a contiguous staging buffer.
//
// The remote prefix cache keeps suspended prefixes' KV in spare memory and
// restores it into the serving cache instead of recomputing the prefix
// (Sec. 6.2.3).  Import scatters staging block i to pool block ids[i] (the
// restore); export gathers pool block ids[i] into staging block i (the
// migration out).  A block is contiguous in both places (16 tokens x Hkv x D
// of one tensor), so either move is a stream of coalesced 16-byte loads and
// stores: one workgroup per (tensor, staging block), each thread moving
// 16-byte vectors, loads batched ahead of stores so several are in flight per
// thread.  Ids outside the pool are skipped and counted.
#include "kernels.h"

namespace specgen {

template <int UNROLL>
__device__ __forceinline__ void copy_block(const uint8_t* src, uint8_t* dst, int64_t bb) {
  if ((bb & 15) == 0) {
    const int64_t nv = bb >> 4;
    const u32x4* s = reinterpret_cast<const u32x4*>(src);
    u32x4* d = reinterpret_cast<u32x4*>(dst);
    for (int64_t base = threadIdx.x; base < nv; base += 256 * UNROLL) {
      u32x4 r[UNROLL];
#pragma unroll
      for (int u = 0; u < UNROLL; ++u) {
        const int64_t e = base + u * 256;
        if (e < nv) r[u] = __builtin_nontemporal_load(s + e);
      }
#pragma unroll
      for (int u = 0; u < UNROLL; ++u) {
        const int64_t e = base + u * 256;
        if (e < nv) __builtin_nontemporal_store(r[u], d + e);
      }
    }
  } else {
    const int64_t nw = bb >> 2;
    const uint32_t* s = reinterpret_cast<const uint32_t*>(src);
    uint32_t* d = reinterpret_cast<uint32_t*>(dst);
    for (int64_t e = threadIdx.x; e < nw; e += 256) d[e] = s[e];
  }
}

// Pool block id of staging block blockIdx.x, or -1 (counted once) if it lies
// outside the pool.
__device__ __forceinline__ int64_t pool_block(const BlockCopyArgs& a) {
  const int64_t id = a.ids[blockIdx.x];
  if (id < 0 || id >= a.num_pool_blocks) {
    if (blockIdx.y == 0 && threadIdx.x == 0 && a.bad_id_count) atomicAdd(a.bad_id_count, 1);
    return -1;
  }
  return id;
}

template <int UNROLL>
__global__ void __launch_bounds__(256) kv_import_kernel(const BlockCopyArgs a) {
  const int64_t id = pool_block(a);
  if (id < 0) return;
  const BlockCopyTensor& T = a.t[blockIdx.y];
  copy_block<UNROLL>(T.staging + (int64_t)blockIdx.x * T.block_bytes, T.pool + id * T.block_bytes, T.block_bytes);
}

template <int UNROLL>
__global__ void __launch_bounds__(256) kv_export_kernel(const BlockCopyArgs a) {
  const int64_t id = pool_block(a);
  if (id < 0) return;
  const BlockCopyTensor& T = a.t[blockIdx.y];
  copy_block<UNROLL>(T.pool + id * T.block_bytes, T.staging + (int64_t)blockIdx.x * T.block_bytes, T.block_bytes);
}

hipError_t launch_kv_import(const BlockCopyArgs& a, hipStream_t stream) {
  if (a.n == 0) return hipSuccess;
  const dim3 grid((unsigned)a.n, (unsigned)a.num_tensors), block(256);
  hipLaunchKernelGGL(kv_import_kernel<8>, grid, block, 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_kv_export(const BlockCopyArgs& a, hipStream_t stream) {
  if (a.n == 0) return hipSuccess;
  const dim3 grid((unsigned)a.n, (unsigned)a.num_tensors), block(256);
  hipLaunchKernelGGL(kv_export_kernel<8>, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace specgen
