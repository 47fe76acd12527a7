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

// ---- the attention kernel's access pattern, without its arithmetic --------
// Tiles as the bf16 partial kernel streams them for head_dim 128: 64 tokens =
// four 16-token pool blocks; per block one kv head's K slice (16 x 128 bf16,
// 4 KiB) and V slice, each moved by one wave as four 1 KiB LDS-DMA pieces;
// eight waves, four 32 KiB LDS stages, three tiles in flight.
constexpr int kRingStages = 4;
constexpr int kSlice = 4096;
constexpr int kRingTile = 8 * kSlice;    // 32 KiB: K and V of four blocks
constexpr int kRingIdCap = 4 * 1024;     // block ids of one worker's tiles

__device__ __forceinline__ void ring_dma(const void* gbase, uint32_t voff, uint32_t lds_addr) {
  const uint64_t g = reinterpret_cast<uint64_t>(gbase);
  const uint32_t glo = __builtin_amdgcn_readfirstlane((uint32_t)g);
  const uint32_t ghi = __builtin_amdgcn_readfirstlane((uint32_t)(g >> 32));
  const void* gu = reinterpret_cast<const void*>(((uint64_t)ghi << 32) | glo);
  const uint32_t l = __builtin_amdgcn_readfirstlane(lds_addr);
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1 nt" ::"v"(voff), "s"(gu), "s"(l) : "m0");
}
template <int N>
__device__ __forceinline__ void ring_wait() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }

// Worker w takes tiles [g0, g0 + n) of the kv_heads * tiles_per_head tiles
// (an even split); tile g is tile k = g % tiles_per_head of kv head g /
// tiles_per_head, whose blocks are table[4k .. 4k + 3].  Waves 0-3 move the K
// slices (wave c: block c of the tile), waves 4-7 the V slices.  Each wave has
// exactly four DMA instructions per tile in flight, so "tile s landed" is
// vmcnt <= 4 x (tiles issued after s).
__global__ void __launch_bounds__(512, 1) slice_ring_kernel(const uint8_t* __restrict__ k_pool,
                                                            const uint8_t* __restrict__ v_pool, int64_t num_blocks,
                                                            int kv_heads, const int32_t* __restrict__ table,
                                                            int tiles_per_head, uint32_t* __restrict__ sink) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kRingStages * kRingTile];
  __shared__ int32_t ids[kRingIdCap];
  const int total = kv_heads * tiles_per_head;
  const int per = total / (int)gridDim.x, rem = total % (int)gridDim.x;
  const int w = blockIdx.x;
  const int g0 = w * per + (w < rem ? w : rem);
  const int n = per + (w < rem ? 1 : 0);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // the block ids of the range, clamped into the pool
  for (int e = tid; e < 4 * n; e += 512) {
    const int g = g0 + e / 4;
    int id = table[4 * (g % tiles_per_head) + (e & 3)];
    id = id < 0 ? 0 : (id >= num_blocks ? (int)(num_blocks - 1) : id);
    ids[e] = id;
  }
  __syncthreads();
  const bool is_v = wave >= 4;
  const int c = wave & 3;
  const int64_t blk_stride = (int64_t)kv_heads * kSlice;
  const uint32_t base = (uint32_t)(size_t)((__attribute__((address_space(3))) uint8_t*)lds);
  auto issue = [&](int s) {
    const int g = g0 + s;
    const int j = g / tiles_per_head;
    const int id = __builtin_amdgcn_readfirstlane(ids[4 * s + c]);
    const uint8_t* src = (is_v ? v_pool : k_pool) + (int64_t)id * blk_stride + (int64_t)j * kSlice;
    const uint32_t st = base + (uint32_t)((s & 3) * kRingTile + (is_v ? 4 * kSlice : 0) + c * kSlice);
#pragma unroll
    for (int i = 0; i < 4; ++i) ring_dma(src, (uint32_t)(i * 1024 + lane * 16), st + (uint32_t)(i * 1024));
  };
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (int s = 0; s < kRingStages - 1 && s < n; ++s) issue(s);
  for (int s = 0; s < n; ++s) {
    if (s + 2 < n) ring_wait<8>();
    else if (s + 1 < n) ring_wait<4>();
    else ring_wait<0>();
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    // the stage of tile s - 1, which every wave finished reading before the barrier
    if (s + kRingStages - 1 < n) issue(s + kRingStages - 1);
    acc ^= *reinterpret_cast<const u32x4*>(lds + (s & 3) * kRingTile + tid * 16);
  }
  if ((acc[0] ^ acc[1] ^ acc[2] ^ acc[3]) == 0x9E3779B9u) sink[0] = 1u;
}

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

extern "C" int specgen_probe_slice_ring(const void* k_pool, const void* v_pool, int64_t num_blocks, int num_kv_heads,
                                        const int32_t* table, int tiles_per_head, int workers, uint32_t* sink,
                                        hipStream_t stream) {
  if (!k_pool || !v_pool || !table || !sink || num_blocks < 1 || num_kv_heads < 1 || tiles_per_head < 1 ||
      workers < 1 || ((uintptr_t)k_pool & 15) || ((uintptr_t)v_pool & 15))
    return 1;
  const int64_t total = (int64_t)num_kv_heads * tiles_per_head;
  if (total > (int64_t)1 << 30 || (total + workers - 1) / workers * 4 > kRingIdCap) return 1;
  hipLaunchKernelGGL(slice_ring_kernel, dim3(workers), dim3(512), 0, stream, static_cast<const uint8_t*>(k_pool),
                     static_cast<const uint8_t*>(v_pool), num_blocks, num_kv_heads, table, tiles_per_head, sink);
  return (int)hipGetLastError();
}
