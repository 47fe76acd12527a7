// kv_append.hip -- per-step append of each fork's new token into its suffix.
//
// Every decode step adds one token to each fork's private continuation, whose
// KV follows the shared reasoning prefix (Sec. 4.2; Sec. 8.7, prefix caching
// paragraph).  Fork f's token takes suffix position pos[f]: block
// suffix_table[suffix_table_off[f] + pos[f]/16], slot pos[f] % 16.  In that
// block, kv head j's K slice is 16 rows of D elements (the token fills row
// slot) and its V slice is D rows of 16 elements (the token fills column slot,
// one element every 16).  One wavefront per (fork, kv head): the lanes read
// the D new elements of K and of V coalesced and write them out; the K row
// stores are contiguous, the V column stores stride 16 elements.  The work is
// a few KB per fork, so the launch is latency-bound, not bandwidth-bound.
#include "kernels.h"

namespace specgen {

template <typename T>
__global__ void __launch_bounds__(256) kv_append_kernel(const AppendArgs a) {
  const int64_t pair = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (pair >= (int64_t)a.num_forks * a.num_kv_heads) return;
  const int lane = threadIdx.x & 63;
  const int f = (int)(pair / a.num_kv_heads);
  const int j = (int)(pair % a.num_kv_heads);
  const int D = a.head_dim;
  // The new elements, the position and the table offsets do not depend on
  // each other: all of them are issued before the first wait, so the only
  // dependent load is the table entry.  kMaxPer covers D <= 1024.
  constexpr int kMaxPer = 16;
  const T* kn = reinterpret_cast<const T*>(a.k_new) + pair * D;
  const T* vn = reinterpret_cast<const T*>(a.v_new) + pair * D;
  T kx[kMaxPer], vx[kMaxPer];
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    const int d = lane + 64 * i;
    if (d < D) {
      kx[i] = kn[d];
      vx[i] = vn[d];
    }
  }
  const int p = a.pos[f];
  const int t0 = a.suffix_table_off[f];
  const int nb = a.suffix_table_off[f + 1] - t0;
  int64_t b = -1;
  if (p >= 0 && p / 16 < nb) b = a.suffix_table[t0 + p / 16];
  if (b < 0 || b >= a.num_blocks) {
    if (j == 0 && lane == 0 && a.bad_count) atomicAdd(a.bad_count, 1);
    return;
  }
  const int slot = p & 15;
  const int64_t head = b * a.num_kv_heads + j;
  T* kd = reinterpret_cast<T*>(a.k_pool) + (head * 16 + slot) * D;
  T* vd = reinterpret_cast<T*>(a.v_pool) + head * D * 16 + slot;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    const int d = lane + 64 * i;
    if (d < D) {
      kd[d] = kx[i];
      vd[(int64_t)d * 16] = vx[i];
    }
  }
}

hipError_t launch_kv_append(const AppendArgs& a, hipStream_t stream) {
  const int64_t pairs = (int64_t)a.num_forks * a.num_kv_heads;
  if (pairs == 0) return hipSuccess;
  const dim3 grid((unsigned)((pairs + 3) / 4)), block(256);
  if (a.elem_bytes == 2)
    hipLaunchKernelGGL(kv_append_kernel<uint16_t>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(kv_append_kernel<uint8_t>, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace specgen
