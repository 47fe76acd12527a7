// probe.hip -- streaming read and copy kernels that measure what HBM delivers
// to plain, perfectly coalesced access (include/specgen_probe.h): the
// ceilings the benchmark reports beside the fork-decode kernels.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/specgen_probe.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kThreads = 256;
constexpr int kUnroll = 8;                       // 16-byte vectors in flight per thread
constexpr int64_t kChunk = (int64_t)kThreads * kUnroll * 16;   // 32 KiB per workgroup iteration

// Workgroups: 8 per compute unit of a 256-CU device, each over a contiguous
// range of whole 32 KiB chunks (the last range may be shorter).
inline int grid_for(int64_t bytes) {
  const int64_t chunks = (bytes + kChunk - 1) / kChunk;
  return (int)(chunks < 2048 ? chunks : 2048);
}

__global__ void __launch_bounds__(kThreads) stream_read_kernel(const u32x4* __restrict__ src, int64_t nvec,
                                                              uint32_t* __restrict__ sink) {
  const int64_t per = (nvec + gridDim.x - 1) / gridDim.x;
  const int64_t lo = (int64_t)blockIdx.x * per;
  const int64_t hi = lo + per < nvec ? lo + per : nvec;
  uint32_t acc = 0;
  for (int64_t base = lo + threadIdx.x; base < hi; base += kThreads * kUnroll) {
    u32x4 r[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t e = base + (int64_t)u * kThreads;
      r[u] = e < hi ? __builtin_nontemporal_load(src + e) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= r[u][0] ^ r[u][1] ^ r[u][2] ^ r[u][3];
  }
  if (acc == 0x9E3779B9u) sink[0] = acc;
}

__global__ void __launch_bounds__(kThreads) stream_copy_kernel(u32x4* __restrict__ dst, const u32x4* __restrict__ src,
                                                              int64_t nvec) {
  const int64_t per = (nvec + gridDim.x - 1) / gridDim.x;
  const int64_t lo = (int64_t)blockIdx.x * per;
  const int64_t hi = lo + per < nvec ? lo + per : nvec;
  for (int64_t base = lo + threadIdx.x; base < hi; base += kThreads * kUnroll) {
    u32x4 r[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t e = base + (int64_t)u * kThreads;
      if (e < hi) r[u] = __builtin_nontemporal_load(src + e);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t e = base + (int64_t)u * kThreads;
      if (e < hi) __builtin_nontemporal_store(r[u], dst + e);
    }
  }
}

bool bad(const void* p, int64_t bytes) { return !p || bytes <= 0 || (bytes & 15) || ((uintptr_t)p & 15); }

}  // namespace

extern "C" int specgen_probe_stream_read(const void* src, int64_t bytes, uint32_t* sink, hipStream_t stream) {
  if (bad(src, bytes) || !sink) return 1;
  hipLaunchKernelGGL(stream_read_kernel, dim3(grid_for(bytes)), dim3(kThreads), 0, stream,
                     static_cast<const u32x4*>(src), bytes / 16, sink);
  return (int)hipGetLastError();
}

extern "C" int specgen_probe_stream_copy(void* dst, const void* src, int64_t bytes, hipStream_t stream) {
  if (bad(src, bytes) || bad(dst, bytes)) return 1;
  hipLaunchKernelGGL(stream_copy_kernel, dim3(grid_for(bytes)), dim3(kThreads), 0, stream, static_cast<u32x4*>(dst),
                     static_cast<const u32x4*>(src), bytes / 16);
  return (int)hipGetLastError();
}
