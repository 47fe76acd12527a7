// kv_import.hip -- block-table-driven restore of cached KV blocks.
//
// The remote prefix cache keeps suspended prefixes' KV in spare memory and
// restores it into the serving cache instead of recomputing the prefix
// (Sec. 6.2.3).  Here the restored copy sits in a contiguous staging buffer
// and every staging block i is scattered to pool block dst[i].  A block is
// contiguous in both places (16 tokens x Hkv x D of one tensor), so the copy is a
// stream of coalesced 16-byte loads and stores: one workgroup per (tensor,
// staging block), each thread moving 16-byte vectors, loads batched ahead of
// stores so several are in flight per thread.  Ids outside the pool are
// skipped and counted.
#include "kernels.h"

namespace specgen {

template <int UNROLL>
__global__ void __launch_bounds__(256) kv_import_kernel(const ImportArgs a) {
  const int64_t i = blockIdx.x;              // staging block
  const int ti = blockIdx.y;                 // tensor
  const int64_t id = a.dst_ids[i];
  if (id < 0 || id >= a.num_dst_blocks) {
    if (ti == 0 && threadIdx.x == 0 && a.bad_id_count) atomicAdd(a.bad_id_count, 1);
    return;
  }
  const ImportTensor& T = a.t[ti];
  const int64_t bb = T.block_bytes;
  const uint8_t* src = T.src + i * bb;
  uint8_t* dst = T.dst + id * bb;
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

hipError_t launch_kv_import(const ImportArgs& a, hipStream_t stream) {
  if (a.n == 0) return hipSuccess;
  const dim3 grid((unsigned)a.n, (unsigned)a.num_tensors), block(256);
  hipLaunchKernelGGL(kv_import_kernel<8>, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace specgen
